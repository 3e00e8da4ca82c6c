// Per-peer deduplicated dispatch and combine.
//
// The peer windows of Appendix D hold one row per routed (token, expert)
// pair; a token with several experts on one peer then crosses to that peer
// several times.  This path sends it once per peer instead (the traffic per
// peer that Section 6.2 balances shrinks by the duplicates):
//
//   moe_layout_dedup   one row per (token, peer) pair, token order per peer
//                      (the layout kernels over peers: each slot reads as
//                      its peer if it is the token's first slot on it, as
//                      unrouted otherwise);
//   moe_dispatch_dedup the dispatch kernel over the pair rows;
//   moe_expand         on the receiving peer: pair rows -> expert-ordered
//                      rows, the layout a per-slot dispatch would have left;
//   moe_combine_local  on the receiving peer: each pair's weighted sum of its
//                      expert outputs, one bf16 row per pair;
//   moe_combine_dedup  on the source: the combine kernel with unit weights
//                      over the pair rows.
//
// The two receiver-side kernels are token-centric and use the byte-balanced
// plan of the per-slot layout.  For each batch of 64/k tokens every lane
// resolves one slot; the slots of a token are then ordered by (peer, slot)
// in LDS so that a peer group is a run: expand loads the pair row once at
// the start of a run and stores it to every slot of the run, the partial
// combine accumulates a run and stores at its end.

#include "dedup.h"

namespace moe {
namespace {

constexpr int kNoKey = 0x7FFFFFFF;   // sort key of an unrouted slot (last)

// Position of slot lj of a token after ordering the token's k slots by
// (key, slot), whether it opens or closes its run of equal keys, and the
// pair row of the run (the first non-negative q among equal keys, in slot
// order).  key/q are the wavefront's LDS rows, the token's slots starting
// at `base`.
__device__ __forceinline__ void order_slot(const int* key, const int* q, int base, int k, int lj,
                                           int my_key, int& spos, bool& first, bool& last,
                                           int& qrun) {
  spos = 0;
  first = true;
  last = true;
  qrun = -1;
  for (int jj = 0; jj < k; ++jj) {
    const int kk = key[base + jj];
    const int qq = q[base + jj];
    const bool same = kk == my_key;
    spos += (kk < my_key || (same && jj < lj)) ? 1 : 0;
    first = first && !(same && jj < lj);
    last = last && !(same && jj > lj);
    if (same && qrun < 0 && qq >= 0) qrun = qq;
  }
}

// VPL: 1 KiB segments held per lane-set; FULL: row bytes == VPL KiB.
// MODE: how the wavefronts take the plan's parts (as dispatch).
template <int VPL, bool FULL, bool SCALES, int MODE>
__global__ __launch_bounds__(kBlock) void expand_kernel(ExpandArgs a) {
  __shared__ int s_key[kWavesPerBlock][kWave];
  __shared__ int s_q[kWavesPerBlock][kWave];
  __shared__ int s_first[kWavesPerBlock][kWave];
  __shared__ uint64_t s_src[kWavesPerBlock][kWave];
  __shared__ uint64_t s_dst[kWavesPerBlock][kWave];
  __shared__ uint64_t s_ssrc[kWavesPerBlock][SCALES ? kWave : 1];
  __shared__ uint64_t s_sdst[kWavesPerBlock][SCALES ? kWave : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int g = uniform(blockIdx.x * kWavesPerBlock + wv);
  const int W = gridDim.x * kWavesPerBlock;
  const uint32_t rb = (uint32_t)a.row_bytes;
  const uint32_t sb = (uint32_t)a.scale_row_bytes;
  const uint32_t sp = (uint32_t)a.scale_pitch;
  const uint32_t l16 = lane * kVecBytes;
  const int k = a.k;
  const int tpb = kWave / k;
  const int lt = lane / k;
  const int lj = lane - lt * k;
  const bool s16 = SCALES && sb % kVecBytes == 0 && sp % kVecBytes == 0 && sp <= kWaveBytes;
  uint32_t st = 0;

  const int T = (int)a.tokens;
  for_each_part<MODE>(a.bound, a.tickets, g, W, lane, [&](int t0, int t1) {
  // token ranges stay inside the batch whatever the plan holds
  t0 = max(t0, 0);
  t1 = min(t1, T);
  for (int tb = t0; tb < t1; tb += tpb) {
    const int te = min(t1, tb + tpb);
    int key = kNoKey, q = -1, p = -1;
    if (lt < tpb && tb + lt < te) {
      const int64_t s = (int64_t)(tb + lt) * k + lj;
      p = a.pos[s];
      if (p >= 0) {
        const int r = a.topk_idx[s] / a.L;
        if ((unsigned)r < (unsigned)a.R) {
          key = r;
          q = a.tok_pos[s];
        } else {
          st |= MOE_STATUS_BAD_INDEX;   // pos and topk_idx disagree: not copied
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    s_key[wv][lane] = key;
    s_q[wv][lane] = q;
    __builtin_amdgcn_wave_barrier();
    if (lt < tpb) {
      int spos, qrun;
      bool first, last;
      order_slot(s_key[wv], s_q[wv], lt * k, k, lj, key, spos, first, last, qrun);
      uint64_t src = 0, dst = 0, ssrc = 0, sdst = 0;
      if (key != kNoKey) {
        const int r = key;
        const int dl = qrun - a.tok_offset[r];
        const int ol = p - a.rank_offset[r];
        if (qrun >= 0 && dl >= 0 && dl < a.dedup_cap[r]) {
          src = a.dedup_x[r] + (uint64_t)dl * rb;
          if (SCALES) ssrc = a.dedup_scales[r] + (uint64_t)dl * sp;
        } else {
          st |= MOE_STATUS_CAPACITY;
        }
        if (ol >= 0 && ol < a.recv_cap[r]) {
          dst = a.recv_x[r] + (uint64_t)ol * rb;
          if (SCALES) sdst = a.recv_scales[r] + (uint64_t)ol * sp;
        } else {
          st |= MOE_STATUS_CAPACITY;
        }
      }
      __builtin_amdgcn_wave_barrier();
      const int at = lt * k + spos;
      s_src[wv][at] = src;
      s_dst[wv][at] = dst;
      s_first[wv][at] = first ? 1 : 0;
      if (SCALES) {
        s_ssrc[wv][at] = ssrc;
        s_sdst[wv][at] = sdst;
      }
    }
    __builtin_amdgcn_wave_barrier();

    for (int t = tb; t < te; ++t) {
      const int l0 = (t - tb) * k;
      for (uint32_t seg = 0; seg < rb; seg += VPL * kWaveBytes) {
        u32x4 v[VPL];
        u32x4 sv = {0u, 0u, 0u, 0u};
        for (int j = 0; j < k; ++j) {
          const uint8_t* sj = reinterpret_cast<const uint8_t*>(readlane64(s_src[wv][l0 + j], 0));
          if (!sj) continue;   // the run's pair row is missing: nothing to copy
          uint8_t* dj = reinterpret_cast<uint8_t*>(readlane64(s_dst[wv][l0 + j], 0));
          if (uniform(s_first[wv][l0 + j])) {
#pragma unroll
            for (int c = 0; c < VPL; ++c) {
              const uint32_t off = seg + c * kWaveBytes + l16;
              if (FULL || off < rb) v[c] = ld16(sj + off);
            }
            if (s16 && seg == 0) {
              const uint8_t* ss = reinterpret_cast<const uint8_t*>(readlane64(s_ssrc[wv][l0 + j], 0));
              sv = l16 < sb ? ld16(ss + l16) : u32x4{0u, 0u, 0u, 0u};
            }
          }
          if (!dj) continue;
#pragma unroll
          for (int c = 0; c < VPL; ++c) {
            const uint32_t off = seg + c * kWaveBytes + l16;
            if (FULL || off < rb) store_row16<VPL>(dj + off, v[c]);
          }
          if (s16 && seg == 0) {
            uint8_t* sd = reinterpret_cast<uint8_t*>(readlane64(s_sdst[wv][l0 + j], 0));
            if (l16 < sp) store_row16<VPL>(sd + l16, sv);
          }
        }
      }
      if (SCALES && !s16) {
        // Other scale-row sizes: one float32 per lane per pass.
        for (uint32_t o = 0; o < sp; o += kWave * 4) {
          const uint32_t off = o + lane * 4;
          uint32_t s4 = 0;
          for (int j = 0; j < k; ++j) {
            const uint8_t* ss = reinterpret_cast<const uint8_t*>(readlane64(s_ssrc[wv][l0 + j], 0));
            if (!ss) continue;
            if (uniform(s_first[wv][l0 + j])) s4 = off < sb ? ld4(ss + off) : 0u;
            uint8_t* sd = reinterpret_cast<uint8_t*>(readlane64(s_sdst[wv][l0 + j], 0));
            if (sd && off < sp) st4(sd + off, s4);
          }
        }
      }
    }
  }
  });
  finish_parts<MODE>(a.tickets, g, W, lane);
  st = wave_or(st);
  if (st && lane == 0) atomicOr(a.status, st);
}

__device__ __forceinline__ void fma8(float (&acc)[8], const u32x4& v, float w) {
  acc[0] = __builtin_fmaf(w, bf16_lo(v.x), acc[0]);
  acc[1] = __builtin_fmaf(w, bf16_hi(v.x), acc[1]);
  acc[2] = __builtin_fmaf(w, bf16_lo(v.y), acc[2]);
  acc[3] = __builtin_fmaf(w, bf16_hi(v.y), acc[3]);
  acc[4] = __builtin_fmaf(w, bf16_lo(v.z), acc[4]);
  acc[5] = __builtin_fmaf(w, bf16_hi(v.z), acc[5]);
  acc[6] = __builtin_fmaf(w, bf16_lo(v.w), acc[6]);
  acc[7] = __builtin_fmaf(w, bf16_hi(v.w), acc[7]);
}

__device__ __forceinline__ u32x4 pack8(const float (&acc)[8]) {
  u32x4 o;
  o.x = pack_bf16x2(acc[0], acc[1]);
  o.y = pack_bf16x2(acc[2], acc[3]);
  o.z = pack_bf16x2(acc[4], acc[5]);
  o.w = pack_bf16x2(acc[6], acc[7]);
  return o;
}

// Per-run weighted sums of one 1 KiB segment: slots are in run order; the
// sum is stored at the run's last slot (dst 0: the pair row is past its
// region, nothing stored) and restarts from +0.  Unused slots read a routed
// row of the token; their data is zeroed bitwise and their weight is 0.
template <int KW>
__device__ __forceinline__ void reduce_runs(const u32x4 (&v)[KW], const float (&wt)[KW],
                                            const uint32_t (&keep)[KW],
                                            uint8_t* const (&dst)[KW], const bool (&last)[KW],
                                            uint32_t off) {
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    u32x4 x = v[j];
    x.x &= keep[j];
    x.y &= keep[j];
    x.z &= keep[j];
    x.w &= keep[j];
    fma8(acc, x, wt[j]);
    if (last[j]) {
      if (dst[j]) st16_stream(dst[j] + off, pack8(acc));
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    }
  }
}

template <int KW>
__device__ __forceinline__ void gather(u32x4 (&v)[KW], const uint8_t* const (&src)[KW],
                                       uint32_t off) {
#pragma unroll
  for (int j = 0; j < KW; ++j) v[j] = ld16_stream(src[j] + off);
}

// KW: slots resolved per token (>= k).
template <int KW>
__global__ __launch_bounds__(kBlock) void combine_local_kernel(LocalArgs a) {
  __shared__ int s_key[kWavesPerBlock][kWave];
  __shared__ int s_q[kWavesPerBlock][kWave];
  __shared__ uint64_t s_src[kWavesPerBlock][kWave + MOE_MAX_K];
  __shared__ uint64_t s_dst[kWavesPerBlock][kWave + MOE_MAX_K];
  __shared__ float s_w[kWavesPerBlock][kWave + MOE_MAX_K];
  __shared__ int s_last[kWavesPerBlock][kWave + MOE_MAX_K];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int g = uniform(blockIdx.x * kWavesPerBlock + wv);
  const int W = gridDim.x * kWavesPerBlock;
  const uint32_t rb = (uint32_t)a.row_bytes;
  const uint32_t l16 = lane * kVecBytes;
  const int k = a.k;
  const int tpb = kWave / k;
  const int lt = lane / k;
  const int lj = lane - lt * k;
  uint32_t st = 0;
  if (lane < MOE_MAX_K) {
    s_src[wv][kWave + lane] = 0;
    s_dst[wv][kWave + lane] = 0;
    s_w[wv][kWave + lane] = 0.0f;
    s_last[wv][kWave + lane] = 0;
  }

  const int T = (int)a.tokens;
  for_each_part<kPartsStatic>(a.bound, nullptr, g, W, lane, [&](int t0, int t1) {
  // token ranges stay inside the batch whatever the plan holds
  t0 = max(t0, 0);
  t1 = min(t1, T);
  for (int tb = t0; tb < t1; tb += tpb) {
    const int te = min(t1, tb + tpb);
    int key = kNoKey, q = -1, p = -1;
    float wl = 0.0f;
    if (lt < tpb && tb + lt < te) {
      const int64_t s = (int64_t)(tb + lt) * k + lj;
      p = a.pos[s];
      if (p >= 0) {
        const int r = a.topk_idx[s] / a.L;
        if ((unsigned)r < (unsigned)a.R) {
          key = r;
          q = a.tok_pos[s];
          wl = a.topk_w[s];
        } else {
          st |= MOE_STATUS_BAD_INDEX;   // pos and topk_idx disagree: not combined
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    s_key[wv][lane] = key;
    s_q[wv][lane] = q;
    __builtin_amdgcn_wave_barrier();
    if (lt < tpb) {
      int spos, qrun;
      bool first, last;
      order_slot(s_key[wv], s_q[wv], lt * k, k, lj, key, spos, first, last, qrun);
      uint64_t src = 0, dst = 0;
      if (key != kNoKey) {
        const int r = key;
        const int il = p - a.rank_offset[r];
        const int pl = qrun - a.tok_offset[r];
        if (il >= 0 && il < a.recv_cap[r])
          src = a.expert_y[r] + (uint64_t)il * rb;
        else
          st |= MOE_STATUS_CAPACITY;
        if (last) {
          if (qrun >= 0 && pl >= 0 && pl < a.part_cap[r])
            dst = a.partial[r] + (uint64_t)pl * rb;
          else
            st |= MOE_STATUS_CAPACITY;
        }
      }
      __builtin_amdgcn_wave_barrier();
      const int at = lt * k + spos;
      s_src[wv][at] = src;
      s_w[wv][at] = src ? wl : 0.0f;
      s_dst[wv][at] = dst;
      s_last[wv][at] = (key != kNoKey && last) ? 1 : 0;
    }
    __builtin_amdgcn_wave_barrier();

    for (int t = tb; t < te; ++t) {
      const int l0 = (t - tb) * k;
      const uint8_t* src[KW];
      uint8_t* dst[KW];
      float wt[KW];
      uint32_t keep[KW];
      bool last[KW];
      uint64_t any = 0;
      bool runs = false;
#pragma unroll
      for (int j = KW - 1; j >= 0; --j) {
        uint64_t sp = readlane64(s_src[wv][l0 + j], 0);
        uint64_t dp = readlane64(s_dst[wv][l0 + j], 0);
        const float w = readlane_f32(s_w[wv][l0 + j], 0);
        const bool lj_ = uniform(s_last[wv][l0 + j]) != 0;
        sp = (j < k) ? sp : 0;
        src[j] = reinterpret_cast<const uint8_t*>(sp);
        dst[j] = reinterpret_cast<uint8_t*>((j < k) ? dp : 0);
        last[j] = (j < k) && lj_;
        runs = runs || last[j];
        wt[j] = sp ? w : 0.0f;
        keep[j] = sp ? 0xFFFFFFFFu : 0u;
        any = sp ? sp : any;
      }
      if (!runs) continue;           // no routed slot
      if (!any) {                    // runs whose expert rows are all missing: +0 rows
        for (uint32_t off = l16; off < rb; off += kWaveBytes) {
#pragma unroll
          for (int j = 0; j < KW; ++j)
            if (last[j] && dst[j]) st16_stream(dst[j] + off, u32x4{0u, 0u, 0u, 0u});
        }
        continue;
      }
#pragma unroll
      for (int j = 0; j < KW; ++j)
        if (!keep[j]) src[j] = reinterpret_cast<const uint8_t*>(any);
      if constexpr (KW >= 32) {
        // 32 slots of gathers fill the registers: one segment at a time
        u32x4 va[KW];
        for (uint32_t o = l16; o < rb; o += kWaveBytes) {
          gather<KW>(va, src, o);
          reduce_runs<KW>(va, wt, keep, dst, last, o);
        }
        continue;
      }
      // Full 1 KiB segments two at a time (the next segment's gathers are
      // issued before the current one is reduced), then the ragged tail.
      const uint32_t nf = rb / kWaveBytes, tail = rb % kWaveBytes;
      u32x4 va[KW], vb[KW];
      uint32_t o = l16;
      if (nf > 0) gather<KW>(va, src, o);
      for (uint32_t s = 0; s + 2 <= nf; s += 2) {
        gather<KW>(vb, src, o + kWaveBytes);
        reduce_runs<KW>(va, wt, keep, dst, last, o);
        if (s + 2 < nf) gather<KW>(va, src, o + 2 * kWaveBytes);
        reduce_runs<KW>(vb, wt, keep, dst, last, o + kWaveBytes);
        o += 2 * kWaveBytes;
      }
      if (nf & 1u) {
        reduce_runs<KW>(va, wt, keep, dst, last, o);
        o += kWaveBytes;
      }
      if (l16 < tail) {
        gather<KW>(va, src, o);
        reduce_runs<KW>(va, wt, keep, dst, last, o);
      }
    }
  }
  });
  st = wave_or(st);
  if (st && lane == 0) atomicOr(a.status, st);
}

template <int VPL, bool SCALES, int MODE>
hipError_t launch_expand_as(const ExpandArgs& a, int waves, bool full, hipStream_t stream) {
  const dim3 grid(waves / kWavesPerBlock), block(kBlock);
  if (full)
    hipLaunchKernelGGL((expand_kernel<VPL, true, SCALES, MODE>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((expand_kernel<VPL, false, SCALES, MODE>), grid, block, 0, stream, a);
  return hipGetLastError();
}

template <int VPL, bool SCALES>
hipError_t launch_expand_vpl(ExpandArgs a, hipStream_t stream) {
  const bool full = a.row_bytes == (int64_t)VPL * kWaveBytes;
  const void* fn =
      full ? reinterpret_cast<const void*>(&expand_kernel<VPL, true, SCALES, kPartsHybrid>)
           : reinterpret_cast<const void*>(&expand_kernel<VPL, false, SCALES, kPartsHybrid>);
  // a token's pair rows are loaded one after another: about half of
  // dispatch's stores are in flight per wavefront
  const int waves =
      copy_waves(fn, (int64_t)(a.k + 1) / 2 * a.row_bytes, kDispatchInFlight, 256);
  // as dispatch: every part claimed at run time when parts are large (a
  // token moves about (k + 1) / 2 pair rows in and k rows out; measured 3%
  // faster at prefill size, 14% slower at decode size), else the claimed
  // half only while a wavefront owns several parts
  if (claim_all_parts(a.tokens, a.row_bytes, a.k + (a.k + 1) / 2 - 1))
    return launch_expand_as<VPL, SCALES, kPartsClaimed>(a, waves, full, stream);
  if (MOE_PLAN_PARTS / waves < 8)
    return launch_expand_as<VPL, SCALES, kPartsStatic>(a, waves, full, stream);
  return launch_expand_as<VPL, SCALES, kPartsHybrid>(a, waves, full, stream);
}

template <bool SCALES>
hipError_t launch_expand_scales(const ExpandArgs& a, hipStream_t stream) {
  const int64_t segs = (a.row_bytes + kWaveBytes - 1) / kWaveBytes;
  switch (segs) {
    case 1: return launch_expand_vpl<1, SCALES>(a, stream);
    case 2: return launch_expand_vpl<2, SCALES>(a, stream);
    case 3: return launch_expand_vpl<3, SCALES>(a, stream);
    case 4: return launch_expand_vpl<4, SCALES>(a, stream);
    case 5: return launch_expand_vpl<5, SCALES>(a, stream);
    case 6: return launch_expand_vpl<6, SCALES>(a, stream);
    case 7: return launch_expand_vpl<7, SCALES>(a, stream);
    case 8: return launch_expand_vpl<8, SCALES>(a, stream);
    case 9: return launch_expand_vpl<9, SCALES>(a, stream);
    case 10: return launch_expand_vpl<10, SCALES>(a, stream);
    case 11: return launch_expand_vpl<11, SCALES>(a, stream);
    case 12: return launch_expand_vpl<12, SCALES>(a, stream);
    case 13: return launch_expand_vpl<13, SCALES>(a, stream);
    case 14: return launch_expand_vpl<14, SCALES>(a, stream);
    case 15: return launch_expand_vpl<15, SCALES>(a, stream);
    default: return launch_expand_vpl<kMaxSegVecs, SCALES>(a, stream);
  }
}

template <int KW>
hipError_t launch_local_kw(LocalArgs a, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&combine_local_kernel<KW>);
  const int waves =
      copy_waves(fn, (KW >= 32 ? 1ll : 2ll) * KW * kWaveBytes, kCombineInFlight, 512);
  hipLaunchKernelGGL((combine_local_kernel<KW>), dim3(waves / kWavesPerBlock), dim3(kBlock), 0,
                     stream, a);
  return hipGetLastError();
}

}  // namespace

DedupGeom dedup_geom(int64_t T, int k, int R) {
  DedupGeom d;
  d.g = layout_geom(T, R);
  d.spare_offset = (d.g.total + 255) / 256 * 256;
  d.total = d.spare_offset + ((size_t)(2 * R + 1) * 4 + 255) / 256 * 256;
  return d;
}

hipError_t launch_expand(const ExpandArgs& a, hipStream_t stream) {
  return a.dedup_scales ? launch_expand_scales<true>(a, stream)
                        : launch_expand_scales<false>(a, stream);
}

hipError_t launch_combine_local(const LocalArgs& a, hipStream_t stream) {
  switch (slot_width(a.k)) {
    case 2: return launch_local_kw<2>(a, stream);
    case 4: return launch_local_kw<4>(a, stream);
    case 8: return launch_local_kw<8>(a, stream);
    case 16: return launch_local_kw<16>(a, stream);
    default: return launch_local_kw<32>(a, stream);
  }
}

}  // namespace moe
