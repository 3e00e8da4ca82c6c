// Dispatch: copy each routed token row into its rank's receive region.
//
// Work split (Section 6.2 with one memory tier, Appendix D third level):
// moe_layout leaves MOE_PLAN_PARTS contiguous token ranges of equal byte
// cost (a token costs one row read plus one row write per routed slot).  The
// kernel launches W wavefronts (a power of two chosen by copy_waves) and
// wavefront g takes parts g, g + W, g + 2W, ...: every wavefront moves the
// same number of bytes no matter how skewed the routing is (a hot expert only
// changes where rows land, not who copies them), and at any moment the W
// wavefronts work on neighbouring parts, so x is read and each expert window
// is written as one advancing front instead of W scattered streams (on
// MI355X that measured ~5% faster for dispatch and ~7% for combine than
// giving each wavefront one contiguous run of parts).  Equal bytes are not
// equal time on a shared memory system, so under the default split parts
// are also handed out at run time from a workspace counter, in plan order
// (the front is kept): every part after each wavefront's first when parts
// are large (kClaimAllPartBytes), the second half of the parts otherwise.
//
// Push direction: a wavefront reads its token's row from x once into
// registers (16 bytes per lane per 1 KiB segment, so a 14 KiB row is 14
// dwordx4 loads in flight per lane) and stores it to each of the token's k
// destinations.  x is read exactly once; every destination row is written
// by exactly one wavefront with full 1 KiB coalesced stores, non-temporal for
// rows wider than 8 KiB (written once, not read again here; with the
// advancing front this measured 8-12% faster than ordinary stores on
// MI355X) and ordinary for narrower rows (store_row16).  Slot metadata
// (pos, expert, region base, capacity) for a batch of 64/k tokens is loaded
// once, one slot per lane, and parked in LDS; the copy loop reads each
// destination back at a uniform LDS address, so no global load of metadata
// (whose wait would also wait for every pending row store) sits between
// row stores.

#include "moe_internal.h"

namespace moe {
namespace {

// VPL: 1 KiB segments held per lane-set (row bytes up to VPL KiB per pass).
// FULL: row bytes == VPL KiB exactly (no per-lane tail test).
template <int VPL, bool FULL, bool SCALES, int MODE>
__global__ __launch_bounds__(kBlock) void dispatch_kernel(DispatchArgs a) {
  // Destination row (and scale row) of every slot of the current batch, one
  // entry per lane of each wavefront (0 = slot not dispatched), padded with
  // zeros so a token can read k entries without a bounds test.
  __shared__ uint64_t s_dst[kWavesPerBlock][kWave + MOE_MAX_K];
  __shared__ uint64_t s_sdst[kWavesPerBlock][SCALES ? kWave + MOE_MAX_K : 1];
  // Per-rank tables (first global row, capacity, region bases), staged once
  // per workgroup: a slot's destination is then an LDS lookup behind its pos
  // and expert loads rather than a second, dependent global load.  Measured
  // on MI355X in whole steps: fp8 dispatch 208.0 -> 206.8 us, large 443.9 ->
  // 443.2, prefill and decode unchanged.
  __shared__ int32_t s_roff[MOE_MAX_EXPERTS];
  __shared__ int32_t s_cap[MOE_MAX_EXPERTS];
  __shared__ uint64_t s_rx[MOE_MAX_EXPERTS];
  __shared__ uint64_t s_rs[SCALES ? MOE_MAX_EXPERTS : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int g = uniform(blockIdx.x * kWavesPerBlock + wv);
  const uint64_t t_start = a.trace ? (uint64_t)wall_clock64() : 0;
  for (int i = threadIdx.x; i < a.R; i += kBlock) {
    s_roff[i] = a.rank_offset[i];
    s_cap[i] = a.recv_cap[i];
    s_rx[i] = a.recv_x[i];
    if (SCALES) s_rs[i] = a.recv_scales[i];
  }
  __syncthreads();
  const int W = gridDim.x * kWavesPerBlock;
  const uint32_t rb = (uint32_t)a.row_bytes;
  const uint32_t sb = (uint32_t)a.scale_row_bytes;
  const uint32_t sp = (uint32_t)a.scale_pitch;
  const uint32_t l16 = lane * kVecBytes;
  const int k = a.k;
  const int tpb = kWave / k;        // tokens whose slots fit one lane each
  const int lt = lane / k;          // this lane's token within a batch
  const int lj = lane - lt * k;     // ... and its slot
  uint32_t st = 0;
  if (lane < MOE_MAX_K) {
    s_dst[wv][kWave + lane] = 0;
    if (SCALES) s_sdst[wv][kWave + lane] = 0;
  }
  // Rows that fit in one pass (row bytes <= VPL KiB) are loaded one token
  // ahead: the next token's row is requested before the current one is
  // stored, so its loads complete while the stores drain instead of after
  // them (loads and stores share one in-order completion counter).
  const bool one_pass = rb <= (uint32_t)(VPL * kWaveBytes);
  const bool s16 = SCALES && sb % kVecBytes == 0 && sp % kVecBytes == 0 && sp <= kWaveBytes;
  u32x4 vn[VPL];
  u32x4 svn = {0u, 0u, 0u, 0u};
  int pre_t = -1;   // token whose row vn holds (-1: none)
  auto load_row = [&](u32x4 (&v)[VPL], u32x4& sv, int t) {
    const uint8_t* src = a.x + (int64_t)t * rb;
#pragma unroll
    for (int c = 0; c < VPL; ++c) {
      const uint32_t off = c * kWaveBytes + l16;
      if (FULL || off < rb) v[c] = ld16(src + off);
    }
    if (s16 && l16 < sb) sv = ld16(a.x_scales + (int64_t)t * sb + l16);
  };

  const int T = (int)a.tokens;
  for_each_part<MODE, true>(a.bound, a.tickets, g, W, lane, [&](int t0, int t1, int next) {
  // Token ranges (and the token read ahead) stay inside the batch whatever
  // the plan holds: a layout whose barrier timed out leaves parts of it
  // unwritten.
  t0 = max(t0, 0);
  t1 = min(t1, T);
  if (next >= T) next = -1;
  for (int tb = t0; tb < t1; tb += tpb) {
    const int te = min(t1, tb + tpb);
    uint64_t dst = 0, sdst = 0;
    if (tb + lt < te) {
      const int64_t s = (int64_t)(tb + lt) * k + lj;
      const int p = a.pos[s];
      if (p >= 0) {
        const int r = a.topk_idx[s] / a.L;
        if ((unsigned)r >= (unsigned)a.R) {
          st |= MOE_STATUS_BAD_INDEX;   // pos and topk_idx disagree: not copied
        } else {
          const int local = p - s_roff[r];
          if (local >= 0 && local < s_cap[r]) {
            dst = s_rx[r] + (uint64_t)local * rb;
            if (SCALES) sdst = s_rs[r] + (uint64_t)local * sp;
          } else {
            st |= MOE_STATUS_CAPACITY;
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    s_dst[wv][lane] = dst;
    if (SCALES) s_sdst[wv][lane] = sdst;
    __builtin_amdgcn_wave_barrier();

    for (int t = tb; t < te; ++t) {
      const int l0 = (t - tb) * k;
      const uint8_t* src = a.x + (int64_t)t * rb;
      const uint8_t* ssrc = SCALES ? a.x_scales + (int64_t)t * sb : nullptr;
      // Scale rows (pitch up to 1 KiB, sizes in 16-byte multiples) move with
      // the row: lane l carries bytes [16 l, 16 l + 16) of the pitched row,
      // scales first, zeros after.
      if (one_pass) {
        u32x4 v[VPL];
        u32x4 sv = {0u, 0u, 0u, 0u};
        if (pre_t == t) {
#pragma unroll
          for (int c = 0; c < VPL; ++c) v[c] = vn[c];
          sv = svn;
        } else {
          load_row(v, sv, t);
        }
        pre_t = t + 1 < t1 ? t + 1 : next;
        if (pre_t >= 0) load_row(vn, svn, pre_t);
        for (int j = 0; j < k; ++j) {
          uint8_t* d = reinterpret_cast<uint8_t*>(readlane64(s_dst[wv][l0 + j], 0));
          if (!d) continue;
#pragma unroll
          for (int c = 0; c < VPL; ++c) {
            const uint32_t off = c * kWaveBytes + l16;
            if (FULL || off < rb) store_row16<VPL>(d + off, v[c]);
          }
          if (s16) {
            uint8_t* sd = reinterpret_cast<uint8_t*>(readlane64(s_sdst[wv][l0 + j], 0));
            if (l16 < sp) store_row16<VPL>(sd + l16, sv);
          }
        }
      } else {
      u32x4 sv = {0u, 0u, 0u, 0u};
      if (s16 && l16 < sb) sv = ld16(ssrc + l16);
      for (uint32_t seg = 0; seg < rb; seg += VPL * kWaveBytes) {
        u32x4 v[VPL];
#pragma unroll
        for (int c = 0; c < VPL; ++c) {
          const uint32_t off = seg + c * kWaveBytes + l16;
          if (FULL || off < rb) v[c] = ld16(src + off);
        }
        for (int j = 0; j < k; ++j) {
          uint8_t* d = reinterpret_cast<uint8_t*>(readlane64(s_dst[wv][l0 + j], 0));
          if (!d) continue;
#pragma unroll
          for (int c = 0; c < VPL; ++c) {
            const uint32_t off = seg + c * kWaveBytes + l16;
            if (FULL || off < rb) store_row16<VPL>(d + off, v[c]);
          }
          if (s16 && seg == 0) {
            uint8_t* sd = reinterpret_cast<uint8_t*>(readlane64(s_sdst[wv][l0 + j], 0));
            if (l16 < sp) store_row16<VPL>(sd + l16, sv);
          }
        }
      }
      }
      if (SCALES && !s16) {
        // Other scale-row sizes: one float32 per lane per pass.
        for (uint32_t o = 0; o < sp; o += kWave * 4) {
          const uint32_t off = o + lane * 4;
          uint32_t s4 = 0;
          if (off < sb) s4 = ld4(ssrc + off);
          for (int j = 0; j < k; ++j) {
            uint8_t* d = reinterpret_cast<uint8_t*>(readlane64(s_sdst[wv][l0 + j], 0));
            if (d && off < sp) st4(d + off, s4);
          }
        }
      }
    }
  }
  });
  finish_parts<MODE>(a.tickets, g, W, lane);
  st = wave_or(st);
  if (st && lane == 0) atomicOr(a.status, st);
  trace_wave(a.trace, a.trace_waves, g, t_start, lane);
}

// Pull dispatch for the partitioning study: a wavefront walks a range of
// global (destination) rows and pulls each row's source token from x.
// POLICY MOE_POLICY_ROWS: the N routed rows are split evenly over the W
// wavefronts.  MOE_POLICY_BY_RANK: wavefronts form R fixed groups of W/R
// and group r splits rank r's rows (a per-peer core assignment that ignores
// how many rows each rank receives).  Per batch of 64 rows, lane l resolves
// row ib+l (source row, destination) into LDS, as the push kernel does.
template <int VPL, bool FULL, bool SCALES, int POLICY>
__global__ __launch_bounds__(kBlock) void dispatch_pull_kernel(DispatchArgs a) {
  __shared__ uint64_t s_src[kWavesPerBlock][kWave];
  __shared__ uint64_t s_dst[kWavesPerBlock][kWave];
  __shared__ uint64_t s_ssrc[kWavesPerBlock][SCALES ? kWave : 1];
  __shared__ uint64_t s_sdst[kWavesPerBlock][SCALES ? kWave : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int g = uniform(blockIdx.x * kWavesPerBlock + wv);
  const uint64_t t_start = a.trace ? (uint64_t)wall_clock64() : 0;
  const int W = gridDim.x * kWavesPerBlock;
  const uint32_t rb = (uint32_t)a.row_bytes;
  const uint32_t sb = (uint32_t)a.scale_row_bytes;
  const uint32_t sp = (uint32_t)a.scale_pitch;
  const uint32_t l16 = lane * kVecBytes;
  int64_t i0 = 0, i1 = 0;
  if (POLICY == MOE_POLICY_ROWS) {
    const int64_t n = a.rank_offset[a.R];
    i0 = n * g / W;
    i1 = n * (g + 1) / W;
  } else {
    const int G = W / a.R;  // the launch makes W a multiple of R
    const int r = g / G, q = g - r * G;
    if (r < a.R) {
      const int64_t b = a.rank_offset[r], n = a.rank_offset[r + 1] - b;
      i0 = b + n * q / G;
      i1 = b + n * (q + 1) / G;
    }
  }
  // rows and their sources stay inside the batch whatever the layout left
  const int64_t n_slots = a.tokens * a.k;
  i0 = max(i0, (int64_t)0);
  i1 = min(i1, n_slots);
  uint32_t st = 0;
  for (int64_t ib = i0; ib < i1; ib += kWave) {
    const int64_t ie = min(i1, ib + kWave);
    uint64_t src = 0, dst = 0, ssrc = 0, sdst = 0;
    if (ib + lane < ie) {
      const int64_t i = ib + lane;
      const int s = a.row_src[i];
      const bool known = s >= 0 && s < n_slots;
      const int t = known ? s / a.k : 0;
      const int r = known ? a.topk_idx[s] / a.L : -1;
      const int64_t local = (unsigned)r < (unsigned)a.R ? i - a.rank_offset[r] : -1;
      if (!known || (unsigned)r >= (unsigned)a.R) {
        st |= MOE_STATUS_BAD_INDEX;
      } else if (local >= 0 && local < a.recv_cap[r]) {
        src = reinterpret_cast<uint64_t>(a.x) + (uint64_t)t * rb;
        dst = a.recv_x[r] + (uint64_t)local * rb;
        if (SCALES) {
          ssrc = reinterpret_cast<uint64_t>(a.x_scales) + (uint64_t)t * sb;
          sdst = a.recv_scales[r] + (uint64_t)local * sp;
        }
      } else {
        st |= MOE_STATUS_CAPACITY;
      }
    }
    __builtin_amdgcn_wave_barrier();
    s_src[wv][lane] = src;
    s_dst[wv][lane] = dst;
    if (SCALES) {
      s_ssrc[wv][lane] = ssrc;
      s_sdst[wv][lane] = sdst;
    }
    __builtin_amdgcn_wave_barrier();
    for (int l = 0; l < (int)(ie - ib); ++l) {
      const uint8_t* sr = reinterpret_cast<const uint8_t*>(readlane64(s_src[wv][l], 0));
      uint8_t* d = reinterpret_cast<uint8_t*>(readlane64(s_dst[wv][l], 0));
      if (!d) continue;
      for (uint32_t seg = 0; seg < rb; seg += VPL * kWaveBytes) {
        u32x4 v[VPL];
#pragma unroll
        for (int c = 0; c < VPL; ++c) {
          const uint32_t off = seg + c * kWaveBytes + l16;
          if (FULL || off < rb) v[c] = ld16(sr + off);
        }
#pragma unroll
        for (int c = 0; c < VPL; ++c) {
          const uint32_t off = seg + c * kWaveBytes + l16;
          if (FULL || off < rb) st16(d + off, v[c]);
        }
      }
      if (SCALES) {
        const uint8_t* ss = reinterpret_cast<const uint8_t*>(readlane64(s_ssrc[wv][l], 0));
        uint8_t* sd = reinterpret_cast<uint8_t*>(readlane64(s_sdst[wv][l], 0));
        for (uint32_t o = 0; o < sp; o += kWave * 4) {
          const uint32_t off = o + lane * 4;
          uint32_t s4 = 0;
          if (off < sb) s4 = ld4(ss + off);
          if (off < sp) st4(sd + off, s4);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
  st = wave_or(st);
  if (st && lane == 0) atomicOr(a.status, st);
  trace_wave(a.trace, a.trace_waves, g, t_start, lane);
}

template <int VPL, bool FULL, bool SCALES, int POLICY>
hipError_t launch_pull(DispatchArgs a, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&dispatch_pull_kernel<VPL, FULL, SCALES, POLICY>);
  int waves = a.launch_waves > 0 ? a.launch_waves : resident_waves(fn, 0);
  if (POLICY == MOE_POLICY_BY_RANK && a.launch_waves == 0) {
    // whole groups per rank, and whole workgroups
    waves = waves / a.R * a.R;
    while (waves > a.R && waves % kWavesPerBlock != 0) waves -= a.R;
    if (waves < a.R || waves % kWavesPerBlock != 0) waves = a.R * kWavesPerBlock;
  }
  hipLaunchKernelGGL((dispatch_pull_kernel<VPL, FULL, SCALES, POLICY>),
                     dim3(waves / kWavesPerBlock), dim3(kBlock), 0, stream, a);
  return hipGetLastError();
}

template <int VPL, bool SCALES, int MODE>
hipError_t launch_push_as(const DispatchArgs& a, int waves, bool full, hipStream_t stream) {
  const dim3 grid(waves / kWavesPerBlock), block(kBlock);
  if (full)
    hipLaunchKernelGGL((dispatch_kernel<VPL, true, SCALES, MODE>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((dispatch_kernel<VPL, false, SCALES, MODE>), grid, block, 0, stream, a);
  return hipGetLastError();
}

template <int VPL, bool SCALES, int MODE>
hipError_t launch_push(DispatchArgs a, hipStream_t stream, bool all_static = false);

template <int VPL, bool SCALES>
hipError_t launch_vpl(DispatchArgs a, int policy, hipStream_t stream) {
  const bool full = a.row_bytes == (int64_t)VPL * kWaveBytes;
  if (policy == MOE_POLICY_ROWS)
    return full ? launch_pull<VPL, true, SCALES, MOE_POLICY_ROWS>(a, stream)
                : launch_pull<VPL, false, SCALES, MOE_POLICY_ROWS>(a, stream);
  if (policy == MOE_POLICY_BY_RANK)
    return full ? launch_pull<VPL, true, SCALES, MOE_POLICY_BY_RANK>(a, stream)
                : launch_pull<VPL, false, SCALES, MOE_POLICY_BY_RANK>(a, stream);
  const int64_t rows = a.rows_hint > 0 ? a.rows_hint : a.k;
  if (policy == MOE_POLICY_DYNAMIC ||
      (policy == MOE_POLICY_BALANCED &&
       claim_all_parts(a.tokens, a.row_bytes, rows, kClaimAllDispatchPartBytes)))
    return launch_push<VPL, SCALES, kPartsClaimed>(a, stream);
  return launch_push<VPL, SCALES, kPartsHybrid>(a, stream, policy == MOE_POLICY_STATIC);
}

template <int VPL, bool SCALES, int MODE>
hipError_t launch_push(DispatchArgs a, hipStream_t stream, bool all_static) {
  const bool full = a.row_bytes == (int64_t)VPL * kWaveBytes;
  const void* fn =
      full ? reinterpret_cast<const void*>(&dispatch_kernel<VPL, true, SCALES, MODE>)
           : reinterpret_cast<const void*>(&dispatch_kernel<VPL, false, SCALES, MODE>);
  const int64_t rows = a.rows_hint > 0 ? a.rows_hint : a.k;
  const int waves = a.launch_waves > 0
                        ? a.launch_waves
                        : copy_waves(fn, rows * a.row_bytes, kDispatchInFlight, 256);
  // The run-time share pays one serialized counter claim per two parts; it
  // only pays off while each wavefront owns several parts.
  if (MODE == kPartsHybrid && (all_static || MOE_PLAN_PARTS / waves < 8))
    return launch_push_as<VPL, SCALES, kPartsStatic>(a, waves, full, stream);
  return launch_push_as<VPL, SCALES, MODE>(a, waves, full, stream);
}

template <bool SCALES>
hipError_t launch_scales(const DispatchArgs& a, int policy, hipStream_t stream) {
  const int64_t segs = (a.row_bytes + kWaveBytes - 1) / kWaveBytes;
  switch (segs) {
    case 1: return launch_vpl<1, SCALES>(a, policy, stream);
    case 2: return launch_vpl<2, SCALES>(a, policy, stream);
    case 3: return launch_vpl<3, SCALES>(a, policy, stream);
    case 4: return launch_vpl<4, SCALES>(a, policy, stream);
    case 5: return launch_vpl<5, SCALES>(a, policy, stream);
    case 6: return launch_vpl<6, SCALES>(a, policy, stream);
    case 7: return launch_vpl<7, SCALES>(a, policy, stream);
    case 8: return launch_vpl<8, SCALES>(a, policy, stream);
    case 9: return launch_vpl<9, SCALES>(a, policy, stream);
    case 10: return launch_vpl<10, SCALES>(a, policy, stream);
    case 11: return launch_vpl<11, SCALES>(a, policy, stream);
    case 12: return launch_vpl<12, SCALES>(a, policy, stream);
    case 13: return launch_vpl<13, SCALES>(a, policy, stream);
    case 14: return launch_vpl<14, SCALES>(a, policy, stream);
    case 15: return launch_vpl<15, SCALES>(a, policy, stream);
    default: return launch_vpl<kMaxSegVecs, SCALES>(a, policy, stream);
  }
}

}  // namespace

hipError_t launch_dispatch(const DispatchArgs& a, int policy, hipStream_t stream) {
  return a.x_scales ? launch_scales<true>(a, policy, stream)
                    : launch_scales<false>(a, policy, stream);
}

}  // namespace moe
