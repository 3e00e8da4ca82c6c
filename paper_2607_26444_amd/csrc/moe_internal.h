// Internal declarations of libmoe (HIP, gfx950).  Kernels live in
// layout.hip, dispatch.hip, combine.hip and expert.hip; api.hip validates
// arguments and calls the launchers declared here.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "moe.h"

namespace moe {

constexpr int kWave = 64;            // CDNA wavefront width
constexpr int kBlock = 256;          // threads per workgroup (4 wavefronts)
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kVecBytes = 16;        // one dwordx4 per lane
constexpr int kWaveBytes = kWave * kVecBytes;  // 1 KiB per wavefront access
constexpr int kMaxSegVecs = 16;      // a wavefront holds up to 16 KiB of a row

// Geometry of the layout pass: tokens are cut into nc chunks of chunk_tokens
// (a multiple of kBlock); each chunk is one workgroup.  The chunk count is
// bounded so that the per-chunk expert count matrix [nc][E] stays small
// enough for every placement workgroup to read all of it.
struct LayoutGeom {
  int64_t chunk_tokens;
  int nc;
  int ncp;              // row pitch of the count matrix: E rounded up to 4
  size_t plan_bytes;    // bound[MOE_PLAN_PARTS + 1], padded to 256 bytes
  size_t ticket_offset; // work tickets: kTicketBlockBytes (three sharded groups, see below)
  size_t gen_offset;    // uint64 generation word of the one-launch layout (end of that block)
  size_t counts_offset;
  size_t counts_bytes;  // int32 [nc][ncp], chunk-major
  size_t sync_offset;   // uint64 arrival flags [nc] of the one-launch layout; 0: none
  size_t total;
};

LayoutGeom layout_geom(int64_t T, int E);

// MOE_OK for hipSuccess; otherwise records the error for
// moe_last_hip_error() and returns MOE_ELAUNCH.
int hip_status(hipError_t err);

// Slot width the layout kernels are compiled for: smallest of 2, 4, 8, 16,
// 32 that is >= k.
int slot_width(int k);

// Wavefronts to launch for a persistent copy kernel: as many as the current
// device keeps resident for `kernel` (compute units x resident blocks per
// unit x 4), rounded down to a divisor of MOE_PLAN_PARTS that is a multiple
// of kWavesPerBlock.  Queried once per (device, kernel) and cached.
int resident_waves(const void* kernel, size_t lds_bytes);

// Wavefronts for a byte-balanced copy kernel with `per_wave` bytes of memory
// operations in flight per wavefront: the power of two nearest to
// target / per_wave, between min_waves (a power of two) and the resident
// count.  Each wavefront
// takes every W-th part of the plan, so the W wavefronts sweep the tokens as
// one front.  On MI355X, whole workgroups spread evenly over the compute
// units and a front of about 64 MiB of dispatch stores (16 MiB of combine
// gathers, twice that for decode-sized batches whose parts are small) in
// flight measured fastest over a range of preceding work; in a whole
// layout -> dispatch -> combine step a 32 MiB dispatch front (half the
// wavefronts) is 44-63% slower and a 128 MiB one ~4% slower.
int copy_waves(const void* kernel, int64_t per_wave, int64_t target, int min_waves);
constexpr int64_t kDispatchInFlight = 64ll << 20;
constexpr int64_t kCombineInFlight = 16ll << 20;

// The default split (MOE_POLICY_BALANCED) of combine and expand hands every
// part out at run time when a part carries at least this many algorithmic
// bytes on average (tokens * row bytes * (1 + rows per token) /
// MOE_PLAN_PARTS).  Measured on MI355X with a fresh x per step: claiming
// every part made combine 2-4% faster at 168-192 KiB per part (prefill,
// large, fp8 combine) and, even with sharded tickets, 19% slower at 42 KiB
// (decode: 104.5 vs 87.8 us), where one claim serves a third of a token.
constexpr int64_t kClaimAllPartBytes = 128ll << 10;

// Dispatch (per-slot rows and the per-peer path's pair rows) claims every
// part from half that size.  With sharded tickets, claiming every part
// measured 1.8% faster for the fp8 workload's 84 KiB parts (215 vs 219 us)
// and tied at decode size (42 KiB, which keeps the half-claimed split);
// pair rows measured 4% faster at 93 KiB per part (Zipf-skewed prefill)
// and 0.6% at 107 KiB, where the same split of the source-side sum was 2-5%
// slower and stays at the default.
constexpr int64_t kClaimAllDispatchPartBytes = 64ll << 10;

__host__ __forceinline__ bool claim_all_parts(int64_t tokens, int64_t row_bytes, int64_t rows,
                                              int64_t min_part_bytes = kClaimAllPartBytes) {
  return tokens * row_bytes * (1 + rows) / MOE_PLAN_PARTS >= min_part_bytes;
}

// fixed_cap < 0: packed layout; >= 0: fixed windows of fixed_cap rows.
// peer_L > 0: topk_idx holds experts in [0, E * peer_L) and the layout is
// over the E peers, one row per (token, peer) pair (first slot of the pair).
hipError_t launch_layout(const int32_t* topk_idx, int64_t T, int k, int E, int R,
                         int fixed_cap, int32_t* expert_count, int32_t* expert_offset,
                         int32_t* rank_count, int32_t* rank_offset, int32_t* pos,
                         int32_t* row_src, void* workspace, uint32_t* status,
                         hipStream_t stream, int peer_L = 0);

struct DispatchArgs {
  const uint8_t* x;
  const uint8_t* x_scales;     // nullptr for bf16 payloads
  int64_t tokens;              // T
  int64_t row_bytes;           // 2H (bf16) or H (fp8)
  int32_t scale_row_bytes;     // (H/128)*4 or 0
  int32_t scale_pitch;         // bytes between scale rows of a region (>= scale_row_bytes)
  int32_t k;
  int32_t L;                   // experts per rank
  const int32_t* topk_idx;
  const int32_t* pos;
  const int32_t* rank_offset;
  const uint64_t* recv_x;
  const uint64_t* recv_scales;
  const int32_t* recv_cap;
  const int32_t* bound;        // plan: bound[MOE_PLAN_PARTS + 1]
  int32_t launch_waves;        // wavefronts to launch; 0 = copy_waves' choice
  int32_t rows_hint;           // rows written per token (0: k); > 0: pair rows
  uint32_t* status;
  const int32_t* row_src;      // pull policies only
  int32_t R;
  uint32_t* tickets;           // dynamic policy: {next, done}, zeroed by the layout
  uint64_t* trace;             // optional per-wavefront (start, end) times
  int32_t trace_waves;
};

hipError_t launch_dispatch(const DispatchArgs& a, int policy, hipStream_t stream);

struct CombineArgs {
  const uint64_t* expert_y;
  const float* topk_w;         // nullptr: every weight is 1
  int64_t tokens;              // T
  int64_t row_bytes;           // 2H
  int32_t k;
  int32_t L;
  const int32_t* topk_idx;
  const int32_t* pos;
  const int32_t* rank_offset;
  const int32_t* recv_cap;
  uint16_t* y;
  const int32_t* bound;
  int32_t launch_waves;
  int32_t rows_hint;           // rows gathered per token, for copy_waves (0: all KW)
  uint32_t* status;
  uint64_t* trace;
  int32_t trace_waves;
  uint32_t* tickets;           // dynamic policy: {next, done}, zeroed by the layout
  int32_t R;                   // ranks (entries of expert_y, rank_offset, recv_cap)
};

hipError_t launch_combine(const CombineArgs& a, int policy, hipStream_t stream);

struct ExpertArgs {
  const uint64_t* recv_x;
  const uint64_t* recv_scales;
  int32_t scale_pitch;
  int32_t H;
  int32_t E;
  int32_t L;
  int32_t identity;
  const int32_t* expert_offset;
  const int32_t* rank_offset;
  const int32_t* recv_cap;
  const uint64_t* out_y;
  int64_t max_rows;
};

hipError_t launch_expert_scale(const ExpertArgs& a, bool fp8, hipStream_t stream);

// ---------------------------------------------------------------- device
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) u32x4 gu32x4;
typedef __attribute__((address_space(1))) uint32_t gu32;

// 16-byte and 4-byte accesses to global memory.  Addresses built from
// integers (region tables, readlane) would otherwise compile to flat
// instructions, which also count against the scalar/LDS wait counter.
__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *(const gu32x4*)(uintptr_t)p;
}
__device__ __forceinline__ void st16(void* p, u32x4 v) { *(gu32x4*)(uintptr_t)p = v; }
// Streaming accesses to data touched once: the non-temporal hint keeps it
// from displacing reusable lines (measured on MI355X: 16-byte streaming reads
// go from ~6.2 to ~7.0 TB/s with it).
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load((const gu32x4*)(uintptr_t)p);
}
__device__ __forceinline__ void st16_stream(void* p, u32x4 v) {
  __builtin_nontemporal_store(v, (gu32x4*)(uintptr_t)p);
}
// Row stores of the copy kernels (dispatch, expand), VPL KiB per pass:
// non-temporal for rows of more than 8 KiB, ordinary for narrower rows.
// Measured in whole steps on MI355X: non-temporal stores are 8-12% faster
// for dispatch's 14 KiB rows (prefill, decode), ordinary stores 4% faster
// for the fp8 workload's 7 KiB rows (211 vs 220 us) and 2.5% for the 8 KiB
// rows of the large workload (444 vs 455 us); in the per-peer chain,
// ordinary stores made expand 6% faster for those rows (fp8 445 -> 418 us,
// large 668 -> 635) and the pair dispatch after it 8-10% slower, 0.5% less
// for the chain.
template <int VPL>
__device__ __forceinline__ void store_row16(void* p, u32x4 v) {
  if constexpr (VPL > 8)
    st16_stream(p, v);
  else
    st16(p, v);
}
__device__ __forceinline__ uint32_t ld4(const void* p) { return *(const gu32*)(uintptr_t)p; }
__device__ __forceinline__ void st4(void* p, uint32_t v) { *(gu32*)(uintptr_t)p = v; }

// Buffer resources (base, range in bytes): a load at an offset outside the
// range returns zeros and reads nothing.  Word 3 selects 32-bit untyped data
// on gfx9-family GPUs.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;

// Wavefront-uniform value held in a scalar register.
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Value of lane `l` (wavefront-uniform l) of a 64-bit per-lane value.
__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ float readlane_f32(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// Work tickets.  Each copy kernel that hands parts out at run time (dispatch,
// combine, expand) has a group of kTicketShards counters, each {next claim,
// wavefronts done} on its own 128-byte line; group k starts at word
// k * kTicketGroupWords of the ticket block.  On MI355X device-scope atomics
// on one address serialize at ~13 ns each: one counter for all wavefronts
// capped dispatch at ~80 claims per microsecond (claiming every part at
// decode size was bound by that alone) and made a thousand wavefronts that
// reach their first claim together wait ~25 us.  With each shard spread over
// all XCDs (below), 4 shards measured best of 1, 4, 8 and 16 at every
// workload: whole steps 0.3-0.8% faster than one counter, mostly in combine.
constexpr int kTicketShards = 4;
constexpr int kTicketStride = 32;                                  // words (128 bytes)
// Wavefronts are given to shards in runs of kShardSpan = 32 (eight
// workgroups, which the hardware places on the eight XCDs in turn), so every
// shard draws wavefronts from every XCD and the shards advance at the same
// rate; a shard of wavefronts from one or two XCDs fell behind the others.
constexpr int kShardSpan = 32;

// Shards a launch of W wavefronts uses: one per run of kShardSpan
// wavefronts, at most kTicketShards, so that every shard has wavefronts
// (a shard without any would leave its claims untaken).
__device__ __forceinline__ int ticket_shards(int W) {
  const int n = (W + kShardSpan - 1) / kShardSpan;
  return n < kTicketShards ? n : kTicketShards;
}

__device__ __forceinline__ int ticket_shard(int g, int W) {
  return (g / kShardSpan) % ticket_shards(W);
}

// Number of wavefronts g < W with ticket_shard(g, W) == s.
__device__ __forceinline__ int waves_in_shard(int s, int W) {
  const int ns = ticket_shards(W);
  const int runs = W / kShardSpan, rem = W % kShardSpan;
  int n = (runs / ns + (runs % ns > s ? 1 : 0)) * kShardSpan;
  if (rem && runs % ns == s) n += rem;
  return n;
}
constexpr int kTicketGroupWords = 16 * kTicketStride;              // 2 KiB per kernel (<= 16 shards)
constexpr int kTicketGroups = 3;                                   // dispatch, combine, expand
constexpr size_t kTicketBlockBytes = 8192;                         // groups + generation word
static_assert(kTicketGroups * kTicketGroupWords * 4 + 128 <= (int)kTicketBlockBytes, "tickets");

// How a copy kernel's wavefronts take the parts of the plan.
//   kPartsStatic  wavefront g of W takes parts g, g + W, g + 2W, ...
//   kPartsClaimed wavefront g takes part g, then claims the next unclaimed
//                 part, one at a time, from a ticket counter in the workspace
//   kPartsHybrid  the first half of the parts as kPartsStatic, the rest
//                 claimed two at a time
// Claimed parts come in plan order, so the wavefronts still sweep the tokens
// as one front; claiming lets fast wavefronts take over the tail of slow
// ones without waiting on anyone.  Wavefront g claims from shard
// ticket_shard(g, W) of its kernel's ticket group: claim c of shard s is the
// (c * n + s)-th claim of the plan (n = shards in use), so the shards
// interleave in plan order and each is shared by 1/n of the wavefronts.  moe_layout zeroes the counters and the
// last wavefront of each shard resets that shard for the next launch.
constexpr int kPartsStatic = 0;
constexpr int kPartsClaimed = 1;
constexpr int kPartsHybrid = 2;

template <int MODE>
__device__ __forceinline__ void finish_parts(uint32_t* tickets, int g, int W, int lane) {
  if (MODE != kPartsStatic && lane == 0) {
    const int s = ticket_shard(g, W);
    uint32_t* line = tickets + s * kTicketStride;
    if (atomicAdd(&line[1], 1u) == (uint32_t)waves_in_shard(s, W) - 1u) {
      line[0] = 0u;
      line[1] = 0u;
    }
  }
}

// Calls body(t0, t1) for the token range of every part wavefront g of W
// handles under MODE.  Part boundaries are fetched up to 64 at a time, one
// part per lane, so stepping to the next part (often an empty one when there
// are fewer tokens than parts) costs no global-memory round trip each.
// PEEK: body(t0, t1, next) also gets the first token of the next non-empty
// part this wavefront will take when that is already known (a later part of
// the same fetched group), else -1, so the body can start loading it early.
template <int MODE, bool PEEK = false, typename F>
__device__ __forceinline__ void for_each_part(const int32_t* bound, uint32_t* tickets, int g,
                                              int W, int lane, F&& body) {
  // static share: parts g + i*W below S
  const int S = MODE == kPartsStatic   ? MOE_PLAN_PARTS
                : MODE == kPartsHybrid ? (MOE_PLAN_PARTS / 2) / W * W
                                       : (g < MOE_PLAN_PARTS ? g + 1 : g);
  const int m = MODE == kPartsClaimed ? (g < MOE_PLAN_PARTS ? 1 : 0) : (S - g + W - 1) / W;
  auto call = [&](int b0, int b1, uint64_t nonempty, int i) {
    const int t0 = __builtin_amdgcn_readlane(b0, i), t1 = __builtin_amdgcn_readlane(b1, i);
    if constexpr (PEEK) {
      const uint64_t later = nonempty & ~((2ull << i) - 1ull);   // lanes above i
      const int next = later ? __builtin_amdgcn_readlane(b0, __builtin_ctzll(later)) : -1;
      body(t0, t1, next);
    } else {
      body(t0, t1);
    }
  };
  for (int i0 = 0; i0 < m; i0 += kWave) {
    int b0 = 0, b1 = 0;
    if (i0 + lane < m) {
      const int part = g + (i0 + lane) * W;
      b0 = (int)ld4(bound + part);
      b1 = (int)ld4(bound + part + 1);
    }
    const uint64_t nonempty = PEEK ? __ballot(b0 < b1) : 0ull;
    const int n = m - i0 < kWave ? m - i0 : kWave;
    for (int i = 0; i < n; ++i) call(b0, b1, nonempty, i);
  }
  if (MODE == kPartsStatic) return;
  // claimed share: parts from `first` on, G per claim, from this
  // wavefront's shard (claim c of shard s covers claim c * shards + s)
  constexpr int G = MODE == kPartsHybrid ? 2 : 1;
  const int first = MODE == kPartsHybrid ? S : W;
  const int shards = ticket_shards(W);
  const int shard = ticket_shard(g, W);
  uint32_t* next_claim = tickets + shard * kTicketStride;
  // claims past the last part end the loop (unsigned: a counter that was
  // never reset cannot produce a negative part)
  const int span = MOE_PLAN_PARTS - first;
  const uint32_t n_claims = span > 0 ? (uint32_t)((span + G - 1) / G) : 0u;
  for (;;) {
    uint32_t t = 0;
    if (lane == 0) t = atomicAdd(next_claim, 1u);
    const uint32_t claim =
        (uint32_t)__builtin_amdgcn_readfirstlane((int)t) * (uint32_t)shards + (uint32_t)shard;
    if (claim >= n_claims) break;
    const int p0 = first + (int)claim * G;
    int b0 = 0, b1 = 0;
    if (lane < G && p0 + lane < MOE_PLAN_PARTS) {
      b0 = (int)ld4(bound + p0 + lane);
      b1 = (int)ld4(bound + p0 + lane + 1);
    }
    const uint64_t nonempty = PEEK ? __ballot(b0 < b1) : 0ull;
    const int n = MOE_PLAN_PARTS - p0 < G ? MOE_PLAN_PARTS - p0 : G;
    for (int i = 0; i < n; ++i) call(b0, b1, nonempty, i);
  }
}

// Per-wavefront trace record (start, end) in the constant-rate wall clock.
// The end stamp is taken after the wavefront's stores have completed.
__device__ __forceinline__ void trace_wave(uint64_t* trace, int trace_waves, int g,
                                           uint64_t t_start, int lane) {
  if (trace && g < trace_waves) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    const uint64_t t_end = (uint64_t)wall_clock64();
    if (lane == 0) {
      trace[2 * g] = t_start;
      trace[2 * g + 1] = t_end;
    }
  }
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v |= __shfl_xor(v, d, kWave);
  return v;
}

// bf16 <-> float32.  bf16 is the upper half of a binary32 pattern; the
// float -> bf16 direction uses gfx950's conversion, which rounds to nearest
// even.
__device__ __forceinline__ float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) |
         ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

}  // namespace moe
