// Combine: y[t] = bf16( sum_j w[t,j] * Y(row of slot j) ).
//
// Token-centric gather-reduce with the same byte-balanced partition as
// dispatch (one wavefront per part of the plan).  Slot metadata for a batch
// of 64/k tokens is resolved once, one slot per lane; for each token the
// wavefront then takes its k source rows and weights from those lanes
// (readlane into scalar registers) and walks
// the output row in 1 KiB segments: every lane issues the k independent
// 16-byte gathers of its segment before it accumulates, keeping k loads per
// lane in flight, multiplies-adds in float32 and stores 8 bf16 values.  Each
// output row has exactly one writer, so the reduction needs no atomics
// (Section 6.1 accumulates on chip and writes back once).
//
// Unused and capacity-dropped slots are redirected to a routed row of the
// same token and masked out of the sum with a select (not a multiply by 0,
// which would turn an Inf in that row into NaN).

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

// KW: slots resolved per token (>= k).
template <int KW>
__global__ __launch_bounds__(kBlock) void combine_kernel(CombineArgs a) {
  const int lane = threadIdx.x & (kWave - 1);
  const int part = uniform(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
  if (part >= MOE_PLAN_PARTS) return;
  const int t0 = a.bound[part], t1 = a.bound[part + 1];
  const int64_t rb = a.row_bytes;
  const int k = a.k;
  const int tpb = kWave / k;        // tokens whose slots fit one lane each
  const int lt = lane / k;          // this lane's token within a batch
  const int lj = lane - lt * k;     // ... and its slot
  uint32_t st = 0;

  for (int tb = t0; tb < t1; tb += tpb) {
    const int te = min(t1, tb + tpb);
    // Source row and weight of slot (tb + lt, lj), resolved once per batch.
    uint64_t srow = 0;
    float wl = 0.0f;
    bool ok = false;
    if (tb + lt < te) {
      const int64_t s = (int64_t)(tb + lt) * k + lj;
      const int p = a.pos[s];
      if (p >= 0) {
        const int r = a.topk_idx[s] / a.L;
        const int local = p - a.rank_offset[r];
        if (local >= 0 && local < a.recv_cap[r]) {
          srow = a.expert_y[r] + (uint64_t)local * (uint64_t)rb;
          wl = a.topk_w[s];
          ok = true;
        } else {
          st |= MOE_STATUS_CAPACITY;
        }
      }
    }
    const uint64_t okm = __ballot(ok);

    for (int t = tb; t < te; ++t) {
      const int l0 = (t - tb) * k;
      const uint8_t* src[KW];
      float wt[KW];
      bool use[KW];
      const uint8_t* any = nullptr;
#pragma unroll
      for (int j = 0; j < KW; ++j) {
        src[j] = nullptr;
        wt[j] = 0.0f;
        use[j] = j < k && ((okm >> (l0 + j)) & 1ull);
        if (use[j]) {
          src[j] = reinterpret_cast<const uint8_t*>(readlane64(srow, l0 + j));
          wt[j] = readlane_f32(wl, l0 + j);
          if (!any) any = src[j];
        }
      }
      uint8_t* dst = reinterpret_cast<uint8_t*>(a.y) + (int64_t)t * rb;
      if (!any) {  // no routed slot: y = +0
        for (int64_t off = lane * kVecBytes; off < rb; off += kWaveBytes)
          st16(dst + off, u32x4{0u, 0u, 0u, 0u});
        continue;
      }
#pragma unroll
      for (int j = 0; j < KW; ++j)
        if (!use[j]) src[j] = any;

#pragma unroll 2
      for (int64_t seg = 0; seg < rb; seg += kWaveBytes) {
        const int64_t off = seg + lane * kVecBytes;
        if (off < rb) {
          u32x4 v[KW];
#pragma unroll
          for (int j = 0; j < KW; ++j) v[j] = ld16(src[j] + off);
          float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int j = 0; j < KW; ++j)
            if (use[j]) fma8(acc, v[j], wt[j]);
          u32x4 o;
          o.x = pack_bf16x2(acc[0], acc[1]);
          o.y = pack_bf16x2(acc[2], acc[3]);
          o.z = pack_bf16x2(acc[4], acc[5]);
          o.w = pack_bf16x2(acc[6], acc[7]);
          st16(dst + off, o);
        }
      }
    }
  }
  st = wave_or(st);
  if (st && lane == 0) atomicOr(a.status, st);
}

template <int KW>
hipError_t launch_kw(const CombineArgs& a, hipStream_t stream) {
  const dim3 grid(MOE_PLAN_PARTS / kWavesPerBlock), block(kBlock);
  hipLaunchKernelGGL((combine_kernel<KW>), grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_combine(const CombineArgs& a, hipStream_t stream) {
  switch (slot_width(a.k)) {
    case 2: return launch_kw<2>(a, stream);
    case 4: return launch_kw<4>(a, stream);
    case 8: return launch_kw<8>(a, stream);
    case 16: return launch_kw<16>(a, stream);
    default: return launch_kw<32>(a, stream);
  }
}

}  // namespace moe
