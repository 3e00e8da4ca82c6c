// Stand-in expert used between dispatch and combine by tests and the
// benchmark (not part of the operator): expert e scales its rows by
// s_e = 1 + 0.01*e (or 1), output bf16.  One wavefront per received row.
//
// Every step is a separately rounded float32 operation; contraction into
// fused multiply-adds is switched off so the result is fixed to the bit.

#include "moe_internal.h"

namespace moe {
namespace {

// OCP E4M3FN byte -> float32 (exact): bias 7, subnormals m * 2^-9,
// S.1111.111 is NaN, no infinities.
__device__ __forceinline__ float e4m3_to_f32(uint32_t b) {
  const uint32_t sign = (b & 0x80u) << 24;
  const uint32_t em = b & 0x7Fu;
  if (em == 0x7Fu) return __uint_as_float(sign | 0x7FC00000u);
  const uint32_t ex = em >> 3, m = em & 7u;
  const float mag = ex ? __uint_as_float(((ex + 120u) << 23) | (m << 20))
                       : (float)m * 0x1p-9f;
  return __uint_as_float(__float_as_uint(mag) | sign);
}

template <bool FP8>
__global__ __launch_bounds__(kBlock) void expert_scale_kernel(ExpertArgs a) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t nw = (int64_t)gridDim.x * kWavesPerBlock;
  const int64_t n_rows = a.expert_offset[a.E];
  for (int64_t g = uniform(blockIdx.x * kWavesPerBlock + threadIdx.x / kWave);
       g < n_rows && g < a.max_rows; g += nw) {
    // expert of global row g: last e with expert_offset[e] <= g
    int lo = 0, hi = a.E - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.expert_offset[mid] <= g) lo = mid; else hi = mid - 1;
    }
    const int e = lo, r = e / a.L;
    const int64_t local = g - a.rank_offset[r];
    if (local >= a.recv_cap[r]) continue;
    const float se = a.identity ? 1.0f : 1.0f + 0.01f * (float)e;
    uint8_t* out = reinterpret_cast<uint8_t*>(a.out_y[r]) + local * (int64_t)a.H * 2;
    if (!FP8) {
      const uint8_t* in =
          reinterpret_cast<const uint8_t*>(a.recv_x[r]) + local * (int64_t)a.H * 2;
      for (int64_t off = lane * kVecBytes; off < (int64_t)a.H * 2; off += kWaveBytes) {
        const u32x4 v = ld16(in + off);
        u32x4 o;
        o.x = pack_bf16x2(bf16_lo(v.x) * se, bf16_hi(v.x) * se);
        o.y = pack_bf16x2(bf16_lo(v.y) * se, bf16_hi(v.y) * se);
        o.z = pack_bf16x2(bf16_lo(v.z) * se, bf16_hi(v.z) * se);
        o.w = pack_bf16x2(bf16_lo(v.w) * se, bf16_hi(v.w) * se);
        st16(out + off, o);
      }
    } else {
      const uint8_t* in = reinterpret_cast<const uint8_t*>(a.recv_x[r]) + local * (int64_t)a.H;
      const uint8_t* sc = reinterpret_cast<const uint8_t*>(a.recv_scales[r]) +
                          local * (int64_t)a.scale_pitch;
      // 16 fp8 values per lane; 16 divides 128, so they share one block scale.
      for (int64_t off = lane * kVecBytes; off < a.H; off += kWaveBytes) {
        const u32x4 q = ld16(in + off);
        const float s = __uint_as_float(ld4(sc + (off / MOE_FP8_BLOCK) * 4));
        const uint32_t words[4] = {q.x, q.y, q.z, q.w};
        uint32_t packed[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float f[4];
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const float dq = e4m3_to_f32((words[i] >> (8 * b)) & 0xFFu) * s;
            f[b] = dq * se;
          }
          packed[2 * i] = pack_bf16x2(f[0], f[1]);
          packed[2 * i + 1] = pack_bf16x2(f[2], f[3]);
        }
        st16(out + off * 2, u32x4{packed[0], packed[1], packed[2], packed[3]});
        st16(out + off * 2 + kVecBytes, u32x4{packed[4], packed[5], packed[6], packed[7]});
      }
    }
  }
}

}  // namespace

hipError_t launch_expert_scale(const ExpertArgs& a, bool fp8, hipStream_t stream) {
  int64_t blocks = (a.max_rows + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (fp8)
    hipLaunchKernelGGL(expert_scale_kernel<true>, dim3((unsigned)blocks), dim3(kBlock), 0,
                       stream, a);
  else
    hipLaunchKernelGGL(expert_scale_kernel<false>, dim3((unsigned)blocks), dim3(kBlock), 0,
                       stream, a);
  return hipGetLastError();
}

}  // namespace moe
