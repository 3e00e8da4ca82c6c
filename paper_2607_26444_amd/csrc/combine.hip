// Combine: y[t] = bf16( sum_j w[t,j] * Y(row of slot j) ).
//
// Token-centric gather-reduce with the same byte-balanced partition as
// dispatch (wavefront g of W takes parts g, g + W, ... of the plan; under the
// default split every later part is handed out at run time instead when
// parts are large, kClaimAllPartBytes).  Slot metadata for a batch
// of 64/k tokens is resolved once, one slot per lane, and parked in LDS; for
// each token the wavefront reads its k source rows and weights back at
// uniform LDS addresses (waiting only on the LDS counter, never on pending
// stores) and walks the output row in 1 KiB segments: every lane issues the
// k independent 16-byte gathers of the next segment before it reduces the
// current one and multiplies-adds in float32.  Output rows of 8-16 KiB are
// kept in registers (8 bf16 values per lane and KiB) and stored as one burst
// per token; other widths store each segment as it is reduced.  Each
// output row has exactly one writer, so the reduction needs no atomics
// (Section 6.1 accumulates on chip and writes back once).  Gathers and the
// output stores are non-temporal: every byte is touched once, and on MI355X
// keeping them out of the caches measured fastest for the whole
// dispatch + combine step.
//
// Unused and capacity-dropped slots are redirected to a routed row of the
// same token, their data is zeroed bitwise and their weight is 0 (a plain
// multiply by 0 would turn an Inf in that row into NaN).  When the caller
// expects many unused slots (the source-side sum of the per-peer path, where
// a token's later slots on a peer carry no row), each slot is read through a
// buffer resource instead: an unused slot's resource has an empty range, so
// its loads return +0 without a memory access and need no mask.  That
// measured 8% faster for that sum at Zipf-skewed prefill; with every slot
// routed the redirect measured ~1% faster at decode and is kept there.

#include "moe_internal.h"

namespace moe {
namespace {

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

template <int KW>
__device__ __forceinline__ void gather(u32x4 (&v)[KW], const uint8_t* const (&src)[KW],
                                       uint32_t off) {
#pragma unroll
  for (int j = 0; j < KW; ++j) v[j] = ld16_stream(src[j] + off);
}

// Buffer-resource loads (Rsrc) with cache policy 2, the non-temporal hint.
constexpr int kLoadNonTemporal = 2;

template <int KW>
__device__ __forceinline__ void gather(u32x4 (&v)[KW], const Rsrc (&src)[KW], uint32_t off) {
#pragma unroll
  for (int j = 0; j < KW; ++j)
    v[j] = __builtin_amdgcn_raw_buffer_load_b128(src[j], off, 0, kLoadNonTemporal);
}

// Weighted sum of one 1 KiB segment.  MASKED: unused slots read a routed
// row of the same token; their data is zeroed (bitwise, so an Inf or NaN
// there cannot leak) and their weight is 0.
template <int KW, bool MASKED>
__device__ __forceinline__ u32x4 reduce(const u32x4 (&v)[KW], const float (&wt)[KW],
                                        const uint32_t (&keep)[KW]) {
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    u32x4 x = v[j];
    if (MASKED) {
      x.x &= keep[j];
      x.y &= keep[j];
      x.z &= keep[j];
      x.w &= keep[j];
    }
    fma8(acc, x, wt[j]);
  }
  u32x4 o;
  o.x = pack_bf16x2(acc[0], acc[1]);
  o.y = pack_bf16x2(acc[2], acc[3]);
  o.z = pack_bf16x2(acc[4], acc[5]);
  o.w = pack_bf16x2(acc[6], acc[7]);
  return o;
}

// One token's output row: full 1 KiB segments two at a time, then the
// ragged tail.  The gathers of the next segment are issued before the
// current one is reduced and stored, so waiting for them never waits for a
// store (vector memory operations complete in issue order on this counter).
template <int KW, bool MASKED, typename S>
__device__ __forceinline__ void combine_row(uint8_t* dst, const S (&src)[KW],
                                            const float (&wt)[KW],
                                            const uint32_t (&keep)[KW], uint32_t rb,
                                            uint32_t l16) {
  const uint32_t nf = rb / kWaveBytes, tail = rb % kWaveBytes;
  u32x4 a[KW], b[KW];
  uint32_t o = l16;
  if (nf > 0) gather<KW>(a, src, o);
  for (uint32_t s = 0; s + 2 <= nf; s += 2) {
    gather<KW>(b, src, o + kWaveBytes);
    st16_stream(dst + o, reduce<KW, MASKED>(a, wt, keep));
    if (s + 2 < nf) gather<KW>(a, src, o + 2 * kWaveBytes);
    st16_stream(dst + o + kWaveBytes, reduce<KW, MASKED>(b, wt, keep));
    o += 2 * kWaveBytes;
  }
  if (nf & 1u) {
    st16_stream(dst + o, reduce<KW, MASKED>(a, wt, keep));
    o += kWaveBytes;
  }
  if (l16 < tail) {
    gather<KW>(a, src, o);
    st16_stream(dst + o, reduce<KW, MASKED>(a, wt, keep));
  }
}

// Stores of one output row held in registers (segment s at byte
// l16 + s KiB; lanes past the row end store nothing).
template <int NSEG>
__device__ __forceinline__ void store_row(uint8_t* dst, const u32x4 (&yr)[NSEG], uint32_t rb,
                                          uint32_t l16) {
#pragma unroll
  for (int s = 0; s < NSEG; ++s) {
    const uint32_t o = l16 + (uint32_t)s * kWaveBytes;
    if (o < rb) st16_stream(dst + o, yr[s]);
  }
}

// One token's output row of at most NSEG KiB, reduced into registers
// (ceil(rb / 1 KiB) segments, the last one partial when rb is not a
// multiple of 1 KiB) with the gathers two segments ahead as in combine_row,
// then stored as one burst.  Masked whenever the slots are addressed by
// pointer: the unrolled row is large, and the mask is four ANDs per slot and
// segment (all ones for routed slots).
template <int KW, int NSEG, bool MASKED, typename S>
__device__ __forceinline__ void combine_row_burst(uint8_t* dst, const S (&src)[KW],
                                                  const float (&wt)[KW],
                                                  const uint32_t (&keep)[KW], uint32_t rb,
                                                  uint32_t l16) {
  const uint32_t ns = (rb + kWaveBytes - 1) / kWaveBytes;
  u32x4 v[2][KW], yr[NSEG];
  if (l16 < rb) gather<KW>(v[0], src, l16);
#pragma unroll
  for (int s = 0; s < NSEG; ++s) {
    if ((uint32_t)s < ns) {
      const uint32_t on = l16 + (uint32_t)(s + 1) * kWaveBytes;
      if (on < rb) gather<KW>(v[(s + 1) & 1], src, on);
      yr[s] = reduce<KW, MASKED>(v[s & 1], wt, keep);
    }
  }
  store_row<NSEG>(dst, yr, rb, l16);
}

// KW: slots resolved per token (>= k).  NSEG > 0: rows of at most NSEG KiB,
// each held in registers and stored as one burst (combine_row_burst).  BUF:
// slots read through buffer resources, unused ones with an empty range.
template <int KW, bool DYN, int NSEG, bool BUF>
__global__ __launch_bounds__(kBlock) void combine_kernel(CombineArgs a) {
  // Per-slot source row and weight of the current batch, one entry per lane
  // of each wavefront (0 = slot not combined), padded with zeros so a token
  // can read KW entries without a bounds test.
  __shared__ uint64_t s_src[kWavesPerBlock][kWave + MOE_MAX_K];
  __shared__ float s_w[kWavesPerBlock][kWave + MOE_MAX_K];
  // Under run-time claiming (large parts) the per-rank tables (first global
  // row, capacity, region base) are staged in LDS once per workgroup, so a
  // slot's source row is an LDS lookup behind its pos and expert loads.
  // Measured on MI355X in whole steps: combine 0.25-0.3% faster at prefill,
  // fp8 and large; 0.3-0.6 us slower at decode (static split, 2048
  // wavefronts), which keeps the global loads.
  __shared__ int32_t s_roff[DYN ? MOE_MAX_EXPERTS : 1];
  __shared__ int32_t s_cap[DYN ? MOE_MAX_EXPERTS : 1];
  __shared__ uint64_t s_ry[DYN ? MOE_MAX_EXPERTS : 1];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int g = uniform(blockIdx.x * kWavesPerBlock + wv);
  const uint64_t t_start = a.trace ? (uint64_t)wall_clock64() : 0;
  if constexpr (DYN) {
    for (int i = threadIdx.x; i < a.R; i += kBlock) {
      s_roff[i] = a.rank_offset[i];
      s_cap[i] = a.recv_cap[i];
      s_ry[i] = a.expert_y[i];
    }
    __syncthreads();
  }
  const int W = gridDim.x * kWavesPerBlock;
  const uint32_t rb = (uint32_t)a.row_bytes;
  const uint32_t l16 = lane * kVecBytes;
  const int k = a.k;
  const int tpb = kWave / k;        // tokens whose slots fit one lane each
  const int lt = lane / k;          // this lane's token within a batch
  const int lj = lane - lt * k;     // ... and its slot
  uint32_t st = 0;
  if (lane < MOE_MAX_K) {
    s_src[wv][kWave + lane] = 0;
    s_w[wv][kWave + lane] = 0.0f;
  }

  const int T = (int)a.tokens;
  for_each_part<DYN ? kPartsClaimed : kPartsStatic>(a.bound, a.tickets, g, W, lane,
                                                     [&](int t0, int t1) {
  // token ranges stay inside the batch whatever the plan holds (a layout
  // whose barrier timed out leaves parts of it unwritten)
  t0 = max(t0, 0);
  t1 = min(t1, T);
  for (int tb = t0; tb < t1; tb += tpb) {
    const int te = min(t1, tb + tpb);
    uint64_t srow = 0;
    float wl = 0.0f;
    if (tb + lt < te) {
      const int64_t s = (int64_t)(tb + lt) * k + lj;
      const int p = a.pos[s];
      if (p >= 0) {
        const int r = a.topk_idx[s] / a.L;
        if ((unsigned)r >= (unsigned)a.R) {
          st |= MOE_STATUS_BAD_INDEX;   // pos and topk_idx disagree: weight 0
        } else {
          const int local = p - (DYN ? s_roff[r] : a.rank_offset[r]);
          if (local >= 0 && local < (DYN ? s_cap[r] : a.recv_cap[r])) {
            srow = (DYN ? s_ry[r] : a.expert_y[r]) + (uint64_t)local * (uint64_t)rb;
            wl = a.topk_w ? a.topk_w[s] : 1.0f;   // null: unit weights
          } else {
            st |= MOE_STATUS_CAPACITY;
          }
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
    s_src[wv][lane] = srow;
    s_w[wv][lane] = wl;
    __builtin_amdgcn_wave_barrier();

    for (int t = tb; t < te; ++t) {
      const int l0 = (t - tb) * k;
      const uint8_t* src[KW];
      float wt[KW];
      uint32_t keep[KW];
      uint64_t first = 0;
      bool all = true;
#pragma unroll
      for (int j = KW - 1; j >= 0; --j) {
        uint64_t sp = readlane64(s_src[wv][l0 + j], 0);
        const float w = readlane_f32(s_w[wv][l0 + j], 0);
        sp = (j < k) ? sp : 0;
        src[j] = reinterpret_cast<const uint8_t*>(sp);
        wt[j] = sp ? w : 0.0f;
        keep[j] = sp ? 0xFFFFFFFFu : 0u;
        all = all && sp;
        first = sp ? sp : first;
      }
      uint8_t* dst = reinterpret_cast<uint8_t*>(a.y) + (int64_t)t * rb;
      if (!first) {  // no routed slot: y = +0
        for (uint32_t off = l16; off < rb; off += kWaveBytes)
          st16_stream(dst + off, u32x4{0u, 0u, 0u, 0u});
        continue;
      }
      if (!all) {
#pragma unroll
        for (int j = 0; j < KW; ++j)
          if (!keep[j]) src[j] = reinterpret_cast<const uint8_t*>(first);
      }
      if constexpr (BUF) {
        Rsrc rs[KW];
#pragma unroll
        for (int j = 0; j < KW; ++j)
          rs[j] = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(src[j]), (short)0,
                                                    keep[j] ? (int)rb : 0, kRsrcWord3);
        if constexpr (NSEG > 0) {
          combine_row_burst<KW, NSEG, false>(dst, rs, wt, keep, rb, l16);
        } else {
          combine_row<KW, false>(dst, rs, wt, keep, rb, l16);
        }
      } else if constexpr (NSEG > 0) {
        combine_row_burst<KW, NSEG, true>(dst, src, wt, keep, rb, l16);
      } else if (all) {
        combine_row<KW, false>(dst, src, wt, keep, rb, l16);
      } else {
        combine_row<KW, true>(dst, src, wt, keep, rb, l16);
      }
    }
  }
  });
  finish_parts<DYN ? kPartsClaimed : kPartsStatic>(a.tickets, g, W, lane);
  st = wave_or(st);
  if (st && lane == 0) atomicOr(a.status, st);
  trace_wave(a.trace, a.trace_waves, g, t_start, lane);
}

template <int KW, bool DYN, int NSEG, bool BUF>
hipError_t launch_kw(CombineArgs a, int64_t in_flight, hipStream_t stream) {
  const void* fn = reinterpret_cast<const void*>(&combine_kernel<KW, DYN, NSEG, BUF>);
  // KW gathers of 1 KiB for each of the two segments in flight (of which
  // rows_hint read routed rows when the caller expects masked slots)
  const int64_t rows = a.rows_hint > 0 ? a.rows_hint : KW;
  const int waves = a.launch_waves > 0
                        ? a.launch_waves
                        : copy_waves(fn, 2 * rows * kWaveBytes, in_flight, 512);
  hipLaunchKernelGGL((combine_kernel<KW, DYN, NSEG, BUF>), dim3(waves / kWavesPerBlock),
                     dim3(kBlock), 0, stream, a);
  return hipGetLastError();
}

// Output rows of 8 to 16 KiB (4096 <= H <= 8192 bf16) are stored as one
// burst from registers: on MI355X this measured 2-6% faster at H = 7168 and
// ~1% faster at H = 4096 (where parts are claimed at run time); narrower
// rows, wider rows and slot widths above 8 (whose gathers already fill the
// registers) store each segment as it is reduced.
constexpr int kBurstSegs = 16;

// Buffer-resource slots (BUF) when the caller expects unused slots
// (rows_hint > 0) and the KW resources fit the scalar registers (KW <= 8).
template <int KW, bool DYN, bool BUF>
hipError_t launch_burst(const CombineArgs& a, int64_t in_flight, hipStream_t stream) {
  if (KW <= 8 && a.row_bytes >= 8ll * kWaveBytes &&
      a.row_bytes <= (int64_t)kBurstSegs * kWaveBytes)
    return launch_kw<KW, DYN, (KW <= 8 ? kBurstSegs : 0), BUF>(a, in_flight, stream);
  return launch_kw<KW, DYN, 0, BUF>(a, in_flight, stream);
}

template <int KW, bool DYN>
hipError_t launch_rows(const CombineArgs& a, int64_t in_flight, hipStream_t stream) {
  if constexpr (KW <= 8) {
    if (a.rows_hint > 0) return launch_burst<KW, DYN, true>(a, in_flight, stream);
  }
  return launch_burst<KW, DYN, false>(a, in_flight, stream);
}

template <bool DYN>
hipError_t launch_dyn(const CombineArgs& a, int64_t in_flight, hipStream_t stream) {
  switch (slot_width(a.k)) {
    case 2: return launch_rows<2, DYN>(a, in_flight, stream);
    case 4: return launch_rows<4, DYN>(a, in_flight, stream);
    case 8: return launch_rows<8, DYN>(a, in_flight, stream);
    case 16: return launch_rows<16, DYN>(a, in_flight, stream);
    default: return launch_rows<32, DYN>(a, in_flight, stream);
  }
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, int policy, hipStream_t stream) {
  const int64_t rows = a.rows_hint > 0 ? a.rows_hint : a.k;
  const bool large = claim_all_parts(a.tokens, a.row_bytes, rows);
  const bool claim = policy == MOE_POLICY_DYNAMIC || (policy == MOE_POLICY_BALANCED && large);
  // Small parts (decode-sized batches) measured 2% faster for combine, and
  // the dispatch after it too, with twice the gathers in flight; large
  // parts 6% slower.
  const int64_t in_flight = large ? kCombineInFlight : 2 * kCombineInFlight;
  return claim ? launch_dyn<true>(a, in_flight, stream)
               : launch_dyn<false>(a, in_flight, stream);
}

}  // namespace moe
