// Token placement and partition plan (paper Appendix D, first to third
// level; Section 6.2 for the byte-balanced split).
//
// Two kernels, both one workgroup per chunk of tokens.  A batch of at most
// 256 tokens needs only the second, which then counts for itself; a batch
// of at most kMaxSyncChunks chunks of 256 tokens also runs only the second,
// whose workgroups count their chunks, exchange the counts through the
// workspace and meet at a grid barrier before placing (kPlaceFused):
//
//   layout_count  per-chunk expert histogram.  Each wavefront owns 64
//                 consecutive tokens (one per lane) and sets, for every
//                 routed slot, bit `lane` of an LDS bitmap mask[wave][e]
//                 (ds_or_b64).  The chunk's count for expert e is the sum of
//                 the popcounts of its four wavefront bitmaps.  Bitmap ORs do
//                 not serialize on a hot expert the way counter atomics do,
//                 and the result does not depend on arrival order.
//
// A fixed-capacity variant places expert e's rows in the window
// [e*C, (e+1)*C) instead of after the previous experts' rows.
//
//   layout_place  every chunk reads the whole count matrix (small by
//                 construction, stored chunk-major), derives the global
//                 per-expert totals, their exclusive scan (expert_offset) and
//                 its own prefix over earlier chunks,
//                 then rebuilds its bitmaps and gives each routed slot
//                     pos = expert_offset[e] + (rows of e in earlier chunks)
//                         + (rows of e in earlier sub-chunks of this chunk)
//                         + popcount(bits of e in earlier wavefronts)
//                         + popcount(mask[wave][e] & lanes below this lane).
//                 Since a token routes to an expert at most once, this is the
//                 stable (expert, token) order.  The same pass scans the
//                 per-token cost 1 + (routed slots) and writes the partition
//                 boundaries that fall inside the chunk.
//
// Both kernels decide slot validity with the same routine (load_row), so
// counts and positions always agree.  With peer_L > 0 the same kernels lay
// out one row per (token, peer) pair: E is then the number of peers and
// load_row bins the expert indices by peer as it reads them.

#include <cstdlib>
#include <map>
#include <mutex>
#include <tuple>

#include "moe_internal.h"

namespace moe {
namespace {

// Load token t's k expert indices and decide which slots are routed: an
// index in [0, E) that does not repeat an earlier slot of the row.
// L > 0 (per-peer layout): the indices are experts in [0, E*L), L per peer,
// and each slot becomes its peer e / L if it is the row's first routed slot
// on that peer, else unrouted; the status bits still judge the experts.
template <int KW>
__device__ __forceinline__ void load_row(const int32_t* __restrict__ idx, int64_t t, int64_t T,
                                         int k, int E, int L, int (&ev)[KW], bool (&ok)[KW],
                                         uint32_t& st) {
#pragma unroll
  for (int j = 0; j < KW; ++j) ev[j] = -1;
  if (t < T) {
    if (KW >= 4 && k == KW && (reinterpret_cast<uintptr_t>(idx) & 15) == 0) {
      // the row as 16-byte loads: on MI355X the layout took 0.8-0.9 us less
      // at 4096-32768 tokens than with one 4-byte load per slot
#pragma unroll
      for (int j = 0; j < KW; j += 4) {
        const int4 q = *reinterpret_cast<const int4*>(idx + t * k + j);
        ev[j] = q.x;
        ev[j + 1] = q.y;
        ev[j + 2] = q.z;
        ev[j + 3] = q.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < KW; ++j)
        if (j < k) ev[j] = idx[t * k + j];
    }
  }
  const int n = L > 0 ? E * L : E;
#pragma unroll
  for (int j = 0; j < KW; ++j) {
    const int e = ev[j];
    const bool in_range = e >= 0 && e < n;
    if (e < -1 || e >= n) st |= MOE_STATUS_BAD_INDEX;
    bool repeat = false;
#pragma unroll
    for (int jj = 0; jj < j; ++jj) repeat |= (ev[jj] == e);
    if (in_range && repeat) st |= MOE_STATUS_DUP_INDEX;
    ok[j] = in_range && !repeat;
  }
  if (L > 0) {
    int pr[KW];
#pragma unroll
    for (int j = 0; j < KW; ++j) pr[j] = ok[j] ? ev[j] / L : -1;
#pragma unroll
    for (int j = 0; j < KW; ++j) {
      bool seen = false;
#pragma unroll
      for (int jj = 0; jj < j; ++jj) seen |= (ok[jj] && pr[jj] == pr[j]);
      ev[j] = pr[j];
      ok[j] = ok[j] && !seen;
    }
  }
}

// Inclusive scan over the 64 lanes of a wavefront with gfx9 DPP row shifts
// (within rows of 16 lanes) and row broadcasts (lane 15 into rows 1 and 3,
// then lane 31 into rows 2 and 3).  Lanes a step does not feed add 0.  The
// operands move through the vector ALU, not through LDS as a shuffle does.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Exclusive scans of two uint32 per thread over the 256-thread block (ea,
// eb) and their block totals (ta, tb); the sums must stay below 2^32.
// `scratch` holds 2 * kWavesPerBlock uint32.
__device__ __forceinline__ void block_exclusive_scan2(uint32_t a, uint32_t b, uint32_t* scratch,
                                                      uint32_t& ea, uint32_t& eb, uint32_t& ta,
                                                      uint32_t& tb) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  const uint32_t ia = wave_inclusive_scan(a), ib = wave_inclusive_scan(b);
  if (lane == kWave - 1) {
    scratch[w] = ia;
    scratch[kWavesPerBlock + w] = ib;
  }
  __syncthreads();
  uint32_t ba = 0, bb = 0;
  ta = tb = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    const uint32_t sa = scratch[i], sb = scratch[kWavesPerBlock + i];
    ba += (i < w) ? sa : 0u;
    bb += (i < w) ? sb : 0u;
    ta += sa;
    tb += sb;
  }
  __syncthreads();
  ea = ba + ia - a;
  eb = bb + ib - b;
}

template <int KW>
__global__ __launch_bounds__(kBlock) void layout_count_kernel(
    const int32_t* __restrict__ idx, int64_t T, int k, int E, int peer_L, int64_t chunk_tokens,
    int ncp, int32_t* __restrict__ counts, uint32_t* __restrict__ status) {
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* mask = reinterpret_cast<uint64_t*>(smem);           // [4][E]
  int32_t* cnt = reinterpret_cast<int32_t*>(mask + kWavesPerBlock * E);  // [E]
  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int64_t c0 = (int64_t)blockIdx.x * chunk_tokens;
  const int64_t c1 = min(T, c0 + chunk_tokens);

  for (int i = tid; i < kWavesPerBlock * E; i += kBlock) mask[i] = 0;
  for (int e = tid; e < E; e += kBlock) cnt[e] = 0;
  uint32_t st = 0;
  __syncthreads();

  for (int64_t s0 = c0; s0 < c1; s0 += kBlock) {
    int ev[KW];
    bool ok[KW];
    load_row<KW>(idx, s0 + tid, c1, k, E, peer_L, ev, ok, st);
#pragma unroll
    for (int j = 0; j < KW; ++j)
      if (ok[j]) atomicOr(&mask[w * E + ev[j]], 1ull << lane);
    __syncthreads();
    for (int e = tid; e < E; e += kBlock) {
      int c = 0;
#pragma unroll
      for (int q = 0; q < kWavesPerBlock; ++q) {
        c += __popcll(mask[q * E + e]);
        mask[q * E + e] = 0;
      }
      cnt[e] += c;
    }
    __syncthreads();
  }
  for (int e = tid; e < E; e += kBlock) counts[(int64_t)blockIdx.x * ncp + e] = cnt[e];
  st = wave_or(st);
  if (lane == 0 && st) atomicOr(status, st);
}

constexpr int kMaxExpertsPerThread = MOE_MAX_EXPERTS / kBlock;  // 4
constexpr int kCountBatch = 16;      // 16-byte count loads in flight per thread
constexpr int kMaxCountGroups = 16;  // count-matrix rows read side by side

// How layout_place_kernel learns the per-chunk counts.
//   kPlaceAfterCount  a layout_count launch left the count matrix
//   kPlaceSingle      one workgroup holds the whole batch (T <= kBlock): the
//                     totals are the popcounts of its own bitmaps
//   kPlaceFused       every workgroup counts its chunk (one sub-chunk of
//                     kBlock tokens), publishes its count row, and waits at a
//                     grid barrier until every row is published; one launch
//                     instead of two, and the bitmaps built for counting are
//                     reused for placement
constexpr int kPlaceAfterCount = 0;
constexpr int kPlaceSingle = 1;
constexpr int kPlaceFused = 2;

// The one-launch layout (count, grid barrier, place) serves batches whose
// chunks are single 256-token sub-chunks and whose chunk count is at most
// this; larger grids use the count and place launches.  On MI355X the one
// launch took 11.0 us against 14.3 for two at 16 chunks (decode size) and
// 12.4 against 12.9 at 128 (32768 tokens, 128 experts); at 256 chunks the
// two forms tie.
constexpr int kMaxSyncChunks = 128;

// s_waitcnt operand that waits for every outstanding vector memory operation
// (vmcnt 0) and leaves the other counters free (gfx9 encoding: expcnt 7 in
// bits 6:4, lgkmcnt 15 in bits 11:8, both vmcnt fields 0).
constexpr int kWaitVmcnt0 = 0x0F70;
// Cache policy of a buffer load: sc1, coherent at device (agent) scope.
constexpr int kCoherent = 16;

// Grid barrier of the fused layout without a counter in a known state: the
// workspace holds a generation word and one arrival flag per chunk.  Every
// workgroup reads the generation g at entry and publishes its count row
// with flag = mix(g), then waits until all flags equal mix(g); workgroup 0
// then stores mix(g) as the next generation.  mix is a 64-bit bijection with
// good avalanche (the SplitMix64 finalizer, after adding an odd constant so
// that 0 does not map to 0), so a flag left over from a previous call holds
// an earlier generation's value and cannot match, and memory that was never
// a workspace matches only by a 2^-64 coincidence.  Every call advances the
// word on the device, so a call replayed from a captured graph gets a fresh
// value as well.
//
// Count rows, flags and the generation word are accessed only with
// device-coherent (agent-scope) loads and stores, which on gfx950 bypass the
// compute unit's cache and keep the XCDs' L2 caches coherent for those
// lines.  A workgroup waits until its count-row stores have completed
// before it stores its flag, so a reader that sees the flag and then reads
// the rows with coherent loads sees them complete.  No cache-wide
// write-back or invalidate is needed: on MI355X dropping the release and
// acquire fences (an L2 write-back and an L2 invalidate per workgroup) cut
// the 64-chunk layout from 12.4 to 12.0 us and the 128-chunk one from 12.9
// to 12.4.
__device__ __forceinline__ uint64_t sync_epoch(uint64_t g) {
  uint64_t z = g + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Writes the plan boundaries bound[p] for p in [p_first, p_last], the parts
// that start inside a sub-chunk whose cost units begin at cost_base: part p
// starts at the token after the owner of unit ceil(p*A/P) - 1 (owner[] maps
// the sub-chunk's n_units units to token offsets from s0).  Thread i takes the
// four-part groups i, i + 256, i + 512, ... of the range, so neighbouring
// lanes store neighbouring 16 bytes.  The unit of a part is kept as the
// quotient and remainder of p*A - 1 by P: one division for the thread's
// first group, then steps by A (next part) and by 1024*A (next group of the
// thread), so a single workgroup writing all P + 1 boundaries does no
// division per part.
__device__ __forceinline__ void write_plan(int32_t* __restrict__ bound, int64_t p_first,
                                           int64_t p_last, int64_t A, int64_t cost_base,
                                           int64_t n_units, const uint16_t* owner, int64_t s0) {
  constexpr int64_t P = MOE_PLAN_PARTS;
  constexpr int64_t kStride = 4 * kBlock;    // parts between a thread's groups
  const int64_t q0 = (p_first >> 2) + threadIdx.x;
  const int64_t q_last = p_last >> 2;
  if (q0 > q_last) return;
  // Units (< A <= 2^31), remainders (< P) and the per-step increments fit
  // 32 bits; only the first quotient needs 64-bit arithmetic.
  const int32_t qA = (int32_t)(A / P), rA = (int32_t)(A - (A / P) * P);
  const int32_t qS = (int32_t)(kStride * A / P), rS = (int32_t)(kStride * A - (kStride * A / P) * P);
  // (u, r): floor quotient and remainder of 4q*A - 1 by P for the group's
  // first part p0 = 4q (p0 = 0 gives -1: u = -1, r = P - 1); u is kept
  // relative to the sub-chunk's first unit
  const int64_t n0 = 4 * q0 * A - 1;
  const int64_t u0 = n0 >= 0 ? n0 / P : -1;
  int32_t u = (int32_t)(u0 - cost_base);
  int32_t r = (int32_t)(n0 - u0 * P);
  const int32_t last_unit = (int32_t)n_units - 1;
#pragma unroll 4
  for (int64_t q = q0; q <= q_last; q += kBlock) {
    const int64_t p0 = q * 4;
    int v[4];
    int32_t uu = u, rr = r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // unconditional (clamped) lookup: the four LDS reads go out together
      v[i] = (int)s0 + owner[min(max(uu, 0), last_unit)] + 1;
      uu += qA;
      rr += rA;
      if (rr >= (int32_t)P) {
        rr -= (int32_t)P;
        ++uu;
      }
    }
    if (p0 >= p_first && p0 + 3 <= p_last) {
      *reinterpret_cast<int4*>(bound + p0) = int4{v[0], v[1], v[2], v[3]};
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (p0 + i >= p_first && p0 + i <= p_last) bound[p0 + i] = v[i];
    }
    u += qS;
    r += rS;
    if (r >= (int32_t)P) {
      r -= (int32_t)P;
      ++u;
    }
  }
}

// Sets bound[p] = v for p in [pa, pb]: scalar stores up to a 16-byte
// boundary, then 16-byte stores, then the scalar tail.
constexpr int64_t kFillParts = 1024;   // longest run a thread fills
__device__ __forceinline__ void fill_plan(int32_t* __restrict__ bound, int64_t pa, int64_t pb,
                                          int32_t v) {
  int64_t p = pa;
  for (; p <= pb && (p & 3); ++p) bound[p] = v;
  for (; p + 3 <= pb; p += 4) *reinterpret_cast<int4*>(bound + p) = int4{v, v, v, v};
  for (; p <= pb; ++p) bound[p] = v;
}

// FIXED: fixed-capacity windows of C rows per expert (expert e's window
// starts at e*C); a slot whose rank within its expert reaches C is dropped.
// MODE kPlaceFused: gen, flags and sync_ticks (the barrier's time limit in
// wall-clock ticks; past it the status word gets MOE_STATUS_LAYOUT_SYNC) as
// described at sync_epoch; the counts pointer is then written as well.
template <int KW, int MODE, bool FIXED>
__global__ __launch_bounds__(kBlock) void layout_place_kernel(
    const int32_t* __restrict__ idx, int64_t T, int k, int E, int peer_L, int R, int C,
    int64_t chunk_tokens, int nc, int ncp, int32_t* counts, int32_t* __restrict__ expert_count,
    int32_t* __restrict__ expert_offset, int32_t* __restrict__ rank_count,
    int32_t* __restrict__ rank_offset, int32_t* __restrict__ pos,
    int32_t* __restrict__ row_src, int32_t* __restrict__ bound, uint32_t* __restrict__ tickets,
    uint32_t* __restrict__ status, uint64_t* gen, uint64_t* flags, uint64_t sync_ticks) {
  constexpr bool SINGLE = MODE == kPlaceSingle;
  extern __shared__ __align__(16) unsigned char smem[];
  uint64_t* mask = reinterpret_cast<uint64_t*>(smem);               // [4][E]
  int64_t* scan = reinterpret_cast<int64_t*>(mask + kWavesPerBlock * E);  // [4]
  int32_t* base = reinterpret_cast<int32_t*>(scan + kWavesPerBlock);  // [E]
  int32_t* eoff = base + E;                                         // [E+1]
  int32_t* woff = eoff + E + 1;  // [4][E]; before placement, 2 x [groups][ncp] count partials
  // token (within the sub-chunk) of each cost unit of the sub-chunk
  uint16_t* owner = reinterpret_cast<uint16_t*>(
      woff + (kWavesPerBlock * E > 8 * kBlock ? kWavesPerBlock * E : 8 * kBlock));

  const int tid = threadIdx.x, lane = tid & (kWave - 1), w = tid / kWave;
  const int c = blockIdx.x;
  const int64_t c0 = (int64_t)c * chunk_tokens;
  const int64_t c1 = min(T, c0 + chunk_tokens);
  const int P = MOE_PLAN_PARTS;

  for (int i = tid; i < kWavesPerBlock * E; i += kBlock) mask[i] = 0;

  // The first sub-chunk's indices are requested before the count matrix so
  // both global-memory round trips overlap.
  int ev0[KW];
  bool ok0[KW];
  uint32_t st = 0;
  load_row<KW>(idx, c0 + tid, c1, k, E, peer_L, ev0, ok0, st);

  // Totals and this chunk's prefix for the experts this thread owns:
  // e = tid*EPT .. tid*EPT+EPT-1 (contiguous, so a scan over threads is a
  // scan over experts).
  const int ept = (E + kBlock - 1) / kBlock;
  int tot[kMaxExpertsPerThread], pre[kMaxExpertsPerThread];
  if (MODE != kPlaceAfterCount) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KW; ++j)
      if (ok0[j]) atomicOr(&mask[w * E + ev0[j]], 1ull << lane);
    __syncthreads();
  }
  if constexpr (MODE == kPlaceFused) {
    __shared__ uint32_t s_late;   // this workgroup's wait timed out
    // Publish this chunk's count row, then wait for every chunk's (wave 0
    // alone: one flag per workgroup).
    if (w == 0) {
      const uint64_t epoch =
          sync_epoch(__hip_atomic_load(gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      for (int e = lane; e < E; e += kWave) {
        int cnt = 0;
#pragma unroll
        for (int q = 0; q < kWavesPerBlock; ++q) cnt += __popcll(mask[q * E + e]);
        __hip_atomic_store(counts + (int64_t)c * ncp + e, cnt, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
      // The row's stores complete (vmcnt(0)) before the flag is stored; the
      // signal fences keep the compiler from moving either store across.
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      if (lane == 0)
        __hip_atomic_store(flags + c, epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint64_t t_begin = (uint64_t)wall_clock64();
      for (;;) {
        bool here = true;   // all flags this lane checks (loads issued together)
#pragma unroll
        for (int r = 0; r < (kMaxSyncChunks + kWave - 1) / kWave; ++r) {
          const int i = lane + r * kWave;
          if (i < nc)
            here &= __hip_atomic_load(flags + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                    epoch;
        }
        if (__all(here)) break;
        if ((uint64_t)wall_clock64() - t_begin > sync_ticks) {
          st |= MOE_STATUS_LAYOUT_SYNC;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
      // every workgroup read the generation before it published its flag
      // (advanced after a time-out too, so no flag of this call can pass the
      // next call's barrier)
      if (c == 0 && lane == 0)
        __hip_atomic_store(gen, epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (lane == 0) s_late = (st & MOE_STATUS_LAYOUT_SYNC) ? 1u : 0u;
    }
    // Every wave reads the count matrix after this point, with coherent
    // loads (below).
    __syncthreads();
    if (s_late) {
      // Some chunk's counts did not arrive in time: this chunk places
      // nothing.  Its slots are marked unrouted, so the copy kernels skip
      // them, and the status word carries MOE_STATUS_LAYOUT_SYNC; every
      // workgroup that saw all flags places its chunk from complete counts.
      for (int64_t i = c0 * k + tid; i < c1 * k; i += kBlock) pos[i] = -1;
      if (c == 0 && tid < kTicketGroups * 16 * 2)   // the copy kernels' tickets, as below
        tickets[(tid >> 1) * kTicketStride + (tid & 1)] = 0u;
      st = wave_or(st);
      if (lane == 0 && st) atomicOr(status, st);
      return;
    }
  }
  if (SINGLE) {
#pragma unroll
    for (int q = 0; q < kMaxExpertsPerThread; ++q) {
      tot[q] = pre[q] = 0;
      const int e = tid * ept + q;
      if (q < ept && e < E)
        for (int ww = 0; ww < kWavesPerBlock; ++ww) tot[q] += __popcll(mask[ww * E + e]);
    }
  } else {
    // The count matrix is chunk-major ([nc][ncp], row pitch ncp = E rounded
    // up to 4).  Lanes read neighbouring 16-byte groups of one chunk's row
    // (coalesced), `groups` rows are read side by side, and each thread adds
    // its four experts over every groups-th row with a batch of loads in
    // flight before the first is used.  The groups' partial sums meet in LDS.
    const int q4 = ncp / 4;
    const int groups = min(kBlock / q4, kMaxCountGroups);
    const int gi = tid / q4, li = tid - gi * q4;
    // fused: the rows other workgroups published in this launch, read with
    // device-coherent 16-byte loads through a buffer resource
    const Rsrc rows = __builtin_amdgcn_make_buffer_rsrc(counts, 0, nc * ncp * 4, kRsrcWord3);
    int32_t* part_t = woff;                   // [groups][ncp], free until placement
    int32_t* part_p = woff + groups * ncp;
    if (gi < groups) {
      int4 ta = {0, 0, 0, 0}, pa = {0, 0, 0, 0};
      for (int r0 = gi; r0 < nc; r0 += groups * kCountBatch) {
        int4 v[kCountBatch];
#pragma unroll
        for (int u = 0; u < kCountBatch; ++u) {
          const int r = min(r0 + u * groups, nc - 1);  // past nc: re-read, ignored
          if constexpr (MODE == kPlaceFused) {
            const u32x4 q = __builtin_amdgcn_raw_buffer_load_b128(rows, (r * ncp + li * 4) * 4,
                                                                  0, kCoherent);
            v[u] = int4{(int)q.x, (int)q.y, (int)q.z, (int)q.w};
          } else {
            v[u] = reinterpret_cast<const int4*>(counts + (int64_t)r * ncp)[li];
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // keep every load ahead of the first use
#pragma unroll
        for (int u = 0; u < kCountBatch; ++u) {
          const int r = r0 + u * groups;
          const int in = r < nc ? 1 : 0, before = r < c ? 1 : 0;
          ta.x += in * v[u].x;
          ta.y += in * v[u].y;
          ta.z += in * v[u].z;
          ta.w += in * v[u].w;
          pa.x += before * v[u].x;
          pa.y += before * v[u].y;
          pa.z += before * v[u].z;
          pa.w += before * v[u].w;
        }
      }
      reinterpret_cast<int4*>(part_t + gi * ncp)[li] = ta;
      reinterpret_cast<int4*>(part_p + gi * ncp)[li] = pa;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kMaxExpertsPerThread; ++q) {
      tot[q] = pre[q] = 0;
      const int e = tid * ept + q;
      if (q < ept && e < E)
        for (int g = 0; g < groups; ++g) {
          tot[q] += part_t[g * ncp + e];
          pre[q] += part_p[g * ncp + e];
        }
    }
  }
  // Rows each expert gets: all of its slots, or at most C in fixed windows.
  int64_t my_tot = 0, my_pre = 0;
#pragma unroll
  for (int q = 0; q < kMaxExpertsPerThread; ++q) {
    my_tot += FIXED ? min(tot[q], C) : tot[q];
    my_pre += FIXED ? min(pre[q], C) : pre[q];
  }
  // Both sums are below 2^31 (T * k is).
  uint32_t ex_tot, ex_pre, sum_tot, sum_pre;
  block_exclusive_scan2((uint32_t)my_tot, (uint32_t)my_pre, reinterpret_cast<uint32_t*>(scan),
                        ex_tot, ex_pre, sum_tot, sum_pre);
  int64_t run = ex_tot;                   // rows before my experts
  const int64_t n_total = sum_tot;        // placed rows N
  const int64_t pre_total = sum_pre;      // placed rows before chunk
  // base[e]: window start of expert e (prefix sum, or e*C) plus its rows in
  // earlier chunks; in fixed windows `base - e*C` is the rank within e.
  // eoff[e]: rows placed before expert e (its packed offset), for rank_count.
#pragma unroll
  for (int q = 0; q < kMaxExpertsPerThread; ++q) {
    const int e = tid * ept + q;
    if (q < ept && e < E) {
      const int placed = FIXED ? min(tot[q], C) : tot[q];
      eoff[e] = (int32_t)run;
      base[e] = FIXED ? e * C + pre[q] : (int32_t)(run + pre[q]);
      if (c == 0) {
        expert_count[e] = placed;
        expert_offset[e] = FIXED ? e * C : (int32_t)run;
      }
      run += placed;
    }
  }
  if (tid == 0) eoff[E] = (int32_t)n_total;
  __syncthreads();
  if (c == 0) {
    const int L = E / R;
    if (tid == 0) {
      expert_offset[E] = FIXED ? E * C : (int32_t)n_total;
      rank_offset[R] = FIXED ? E * C : (int32_t)n_total;
      bound[0] = 0;
    }
    // work tickets of dispatch, combine and expand: {next, done} of every shard
    if (tid < kTicketGroups * 16 * 2)   // every line a group can hold
      tickets[(tid >> 1) * kTicketStride + (tid & 1)] = 0u;
    for (int r = tid; r < R; r += kBlock) {
      rank_offset[r] = FIXED ? r * L * C : eoff[r * L];
      rank_count[r] = eoff[(r + 1) * L] - eoff[r * L];
    }
    if (T == 0)
      for (int p = tid; p <= P; p += kBlock) bound[p] = 0;
  }

  // Partition plan: token cost 1 + routed slots, total A = T + N.
  const int64_t A = T + n_total;
  int64_t cost_base = c0 + pre_total;

  for (int64_t s0 = c0; s0 < c1; s0 += kBlock) {
    const int64_t t = s0 + tid;
    int ev[KW];
    bool ok[KW];
    if (s0 == c0) {
#pragma unroll
      for (int j = 0; j < KW; ++j) {
        ev[j] = ev0[j];
        ok[j] = ok0[j];
      }
    } else {
      uint32_t st_more = 0;
      load_row<KW>(idx, t, c1, k, E, peer_L, ev, ok, st_more);
    }
    if (MODE == kPlaceAfterCount) {
#pragma unroll
      for (int j = 0; j < KW; ++j)
        if (ok[j]) atomicOr(&mask[w * E + ev[j]], 1ull << lane);
      __syncthreads();
    }
    // woff[q][e]: first row of expert e for wavefront q of this sub-chunk
    // (base plus the rows of e in wavefronts 0..q-1); base moves past the
    // sub-chunk.  A slot's row is then one lookup plus its rank in its own
    // wavefront's bitmap.
    for (int e = tid; e < E; e += kBlock) {
      int r = base[e];
#pragma unroll
      for (int q = 0; q < kWavesPerBlock; ++q) {
        woff[q * E + e] = r;
        r += __popcll(mask[q * E + e]);
      }
      base[e] = r;
    }
    __syncthreads();
    const uint64_t below = (1ull << lane) - 1ull;
    // Every slot's LDS lookups are issued before any is used (unused slots
    // read expert 0's entries and ignore them): behind a per-slot branch
    // each lookup would wait out its own LDS round trip.
    int rank[KW];
#pragma unroll
    for (int j = 0; j < KW; ++j) {
      const int e = ok[j] ? ev[j] : 0;
      rank[j] = woff[w * E + e] + __popcll(mask[w * E + e] & below);
    }
    int nplaced = 0;
    int pv[KW];
#pragma unroll
    for (int j = 0; j < KW; ++j) {
      pv[j] = -1;
      if (t < c1 && ok[j]) {
        const int r = rank[j];
        if (!FIXED || r - ev[j] * C < C) {
          pv[j] = r;
          row_src[r] = (int32_t)(t * k + j);
          ++nplaced;
        } else {
          st |= MOE_STATUS_CAPACITY;
        }
      }
    }
    if (t < c1) {
      if (k == KW && KW >= 4 && (reinterpret_cast<uintptr_t>(pos) & 15) == 0) {
        // the token's k positions as 16-byte stores
#pragma unroll
        for (int j = 0; j < KW; j += 4)
          *reinterpret_cast<int4*>(pos + t * k + j) = int4{pv[j], pv[j + 1], pv[j + 2], pv[j + 3]};
      } else {
#pragma unroll
        for (int j = 0; j < KW; ++j)
          if (j < k) pos[t * k + j] = pv[j];
      }
    }
    // Plan boundaries inside this sub-chunk: token t owns the parts p with
    // a_t*P < p*A <= (a_t + cost_t)*P, each starting at token t+1.  When no
    // token can own more than kFillParts parts, each thread fills its own
    // token's run (a constant; 16-byte stores inside the run).  Otherwise
    // (batches of a few tokens, where one token may own thousands of parts)
    // the sub-chunk's cost units are mapped to their tokens in LDS and the
    // parts are written part-major (write_plan).  Measured on MI355X for the
    // 128-token, one-workgroup layout: filling runs 0.5 us, part-major 2.6.
    const int64_t cost = (t < c1) ? 1 + nplaced : 0;
    uint32_t ex32, unused_e, sub32, unused_t;
    block_exclusive_scan2((uint32_t)cost, 0u, reinterpret_cast<uint32_t*>(scan), ex32, unused_e,
                          sub32, unused_t);
    const int64_t ex = ex32, sub_total = sub32;
    if ((int64_t)P * (1 + KW) <= kFillParts * A) {
      if (cost > 0)
        fill_plan(bound, ((cost_base + ex) * P) / A + 1, ((cost_base + ex + cost) * P) / A,
                  (int32_t)(t + 1));
    } else {
      for (int64_t u = ex; u < ex + cost; ++u) owner[u] = (uint16_t)tid;
      __syncthreads();
      const int64_t p_first = (cost_base * P) / A + 1;
      const int64_t p_last = ((cost_base + sub_total) * P) / A;
      write_plan(bound, p_first, p_last, A, cost_base, sub_total, owner, s0);
    }
    cost_base += sub_total;
    for (int i = tid; i < kWavesPerBlock * E; i += kBlock) mask[i] = 0;
    __syncthreads();
  }

  if (FIXED) {
    // Window rows no slot fills have no source: for the experts this chunk
    // owns (e = c, c + nc, ...), rows [e*C + placed_e, (e+1)*C).
    for (int e = c; e < E; e += nc) {
      const int placed = eoff[e + 1] - eoff[e];
      for (int i = placed + tid; i < C; i += kBlock) row_src[(int64_t)e * C + i] = -1;
    }
  } else {
    // Rows past the last routed slot have no source.
    for (int64_t i = n_total + (int64_t)c * kBlock + tid; i < T * k; i += (int64_t)nc * kBlock)
      row_src[i] = -1;
  }
  st = wave_or(st);
  if (lane == 0 && st) atomicOr(status, st);
}

// Workgroups of the fused layout that the current device keeps resident at
// once (compute units x resident workgroups per unit for this LDS size),
// queried once per (device, kernel, LDS bytes).  The grid barrier needs every
// workgroup resident.
int resident_blocks(const void* kernel, size_t lds_bytes) {
  static std::mutex mu;
  static std::map<std::tuple<int, const void*, size_t>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(dev, kernel, lds_bytes);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  int cus = 0, blocks = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, kBlock, lds_bytes) !=
          hipSuccess)
    cus = blocks = 0;
  return cache[key] = cus * blocks;
}

// Time limit of the fused layout's grid barrier in wall-clock ticks: 2 s,
// or MOE_LAYOUT_SYNC_LIMIT_US microseconds when that environment variable is
// set (tests of the time-out path), at the current device's wall-clock rate
// (read once per device).
uint64_t sync_limit_ticks() {
  static std::mutex mu;
  static std::map<int, uint64_t> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = -1;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) return it->second;
  int khz = 0;
  if (dev < 0 || hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
      khz < 1)
    khz = 100000;
  uint64_t us = 2000000u;
  if (const char* e = std::getenv("MOE_LAYOUT_SYNC_LIMIT_US")) {
    char* end = nullptr;
    const unsigned long long v = std::strtoull(e, &end, 10);
    if (end != e && v <= 60000000ull) us = v;
  }
  return cache[dev] = (uint64_t)khz * us / 1000u;
}

template <int KW, bool FIXED>
hipError_t launch_layout_kw(const int32_t* idx, int64_t T, int k, int E, int peer_L, int R, int C,
                            int32_t* expert_count, int32_t* expert_offset,
                            int32_t* rank_count, int32_t* rank_offset, int32_t* pos,
                            int32_t* row_src, void* workspace, uint32_t* status,
                            hipStream_t stream) {
  const LayoutGeom g = layout_geom(T, E);
  char* ws = static_cast<char*>(workspace);
  int32_t* bound = reinterpret_cast<int32_t*>(ws);
  int32_t* counts = reinterpret_cast<int32_t*>(ws + g.counts_offset);
  uint32_t* tickets = reinterpret_cast<uint32_t*>(ws + g.ticket_offset);
  uint64_t* gen = reinterpret_cast<uint64_t*>(ws + g.gen_offset);
  uint64_t* flags = g.sync_offset ? reinterpret_cast<uint64_t*>(ws + g.sync_offset) : nullptr;
  const size_t lds_count = (size_t)kWavesPerBlock * E * 8 + (size_t)E * 4;
  // woff also holds the two [groups][ncp] count partials (groups * ncp <=
  // 4 * kBlock int32 each) before placement starts.
  const size_t woff_ints = (size_t)kWavesPerBlock * E > 8 * kBlock ? (size_t)kWavesPerBlock * E
                                                                    : 8 * kBlock;
  const size_t lds_place = (size_t)kWavesPerBlock * E * 8 + kWavesPerBlock * 8 +
                           (size_t)E * 4 + (size_t)(E + 1) * 4 + woff_ints * 4 +
                           (size_t)kBlock * (1 + KW) * 2;
  if (g.nc == 1 && T <= kBlock) {
    hipLaunchKernelGGL((layout_place_kernel<KW, kPlaceSingle, FIXED>), dim3(1), dim3(kBlock),
                       lds_place, stream, idx, T, k, E, peer_L, R, C, g.chunk_tokens, g.nc,
                       g.ncp, counts, expert_count, expert_offset, rank_count, rank_offset, pos,
                       row_src, bound, tickets, status, gen, flags, (uint64_t)0);
    return hipGetLastError();
  }
  const void* fused = reinterpret_cast<const void*>(&layout_place_kernel<KW, kPlaceFused, FIXED>);
  if (flags && g.nc <= resident_blocks(fused, lds_place)) {
    hipLaunchKernelGGL((layout_place_kernel<KW, kPlaceFused, FIXED>), dim3(g.nc), dim3(kBlock),
                       lds_place, stream, idx, T, k, E, peer_L, R, C, g.chunk_tokens, g.nc,
                       g.ncp, counts, expert_count, expert_offset, rank_count, rank_offset, pos,
                       row_src, bound, tickets, status, gen, flags, sync_limit_ticks());
    return hipGetLastError();
  }
  hipLaunchKernelGGL(layout_count_kernel<KW>, dim3(g.nc), dim3(kBlock), lds_count, stream,
                     idx, T, k, E, peer_L, g.chunk_tokens, g.ncp, counts, status);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((layout_place_kernel<KW, kPlaceAfterCount, FIXED>), dim3(g.nc),
                     dim3(kBlock), lds_place, stream, idx, T, k, E, peer_L, R, C,
                     g.chunk_tokens, g.nc, g.ncp, counts, expert_count, expert_offset,
                     rank_count, rank_offset, pos, row_src, bound, tickets, status, gen, flags,
                     (uint64_t)0);
  return hipGetLastError();
}

}  // namespace

LayoutGeom layout_geom(int64_t T, int E) {
  // At most max(1, 32768/E) chunks, each a multiple of kBlock tokens.
  const int64_t nc_max = E >= 32768 ? 1 : 32768 / E;
  const int64_t per = (T + kBlock * nc_max - 1) / (kBlock * nc_max);
  LayoutGeom g;
  g.chunk_tokens = kBlock * (per < 1 ? 1 : per);
  g.nc = (int)((T + g.chunk_tokens - 1) / g.chunk_tokens);
  if (g.nc < 1) g.nc = 1;
  g.ncp = (E + 3) / 4 * 4;
  g.plan_bytes = ((size_t)(MOE_PLAN_PARTS + 1) * 4 + 255) / 256 * 256;
  g.ticket_offset = g.plan_bytes;
  g.gen_offset = g.ticket_offset + kTicketBlockBytes - 128;
  g.counts_offset = g.ticket_offset + kTicketBlockBytes;
  g.counts_bytes = (size_t)g.nc * g.ncp * 4;
  g.total = g.counts_offset + (g.counts_bytes + 255) / 256 * 256;
  g.sync_offset = 0;
  if (g.chunk_tokens == kBlock && g.nc > 1 && g.nc <= kMaxSyncChunks) {
    g.sync_offset = g.total;
    g.total += ((size_t)g.nc * 8 + 255) / 256 * 256;
  }
  return g;
}

int slot_width(int k) {
  int kw = 2;
  while (kw < k) kw *= 2;
  return kw;
}

template <bool FIXED>
hipError_t launch_layout_fx(const int32_t* idx, int64_t T, int k, int E, int peer_L, int R, int C,
                            int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
                            int32_t* rank_offset, int32_t* pos, int32_t* row_src,
                            void* workspace, uint32_t* status, hipStream_t stream) {
  switch (slot_width(k)) {
    case 2:
      return launch_layout_kw<2, FIXED>(idx, T, k, E, peer_L, R, C, expert_count, expert_offset,
                                        rank_count, rank_offset, pos, row_src, workspace,
                                        status, stream);
    case 4:
      return launch_layout_kw<4, FIXED>(idx, T, k, E, peer_L, R, C, expert_count, expert_offset,
                                        rank_count, rank_offset, pos, row_src, workspace,
                                        status, stream);
    case 8:
      return launch_layout_kw<8, FIXED>(idx, T, k, E, peer_L, R, C, expert_count, expert_offset,
                                        rank_count, rank_offset, pos, row_src, workspace,
                                        status, stream);
    case 16:
      return launch_layout_kw<16, FIXED>(idx, T, k, E, peer_L, R, C, expert_count, expert_offset,
                                         rank_count, rank_offset, pos, row_src, workspace,
                                         status, stream);
    default:
      return launch_layout_kw<32, FIXED>(idx, T, k, E, peer_L, R, C, expert_count, expert_offset,
                                         rank_count, rank_offset, pos, row_src, workspace,
                                         status, stream);
  }
}

hipError_t launch_layout(const int32_t* idx, int64_t T, int k, int E, int R, int fixed_cap,
                         int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
                         int32_t* rank_offset, int32_t* pos, int32_t* row_src, void* workspace,
                         uint32_t* status, hipStream_t stream, int peer_L) {
  if (fixed_cap >= 0)
    return launch_layout_fx<true>(idx, T, k, E, peer_L, R, fixed_cap, expert_count,
                                  expert_offset, rank_count, rank_offset, pos, row_src, workspace,
                                  status, stream);
  return launch_layout_fx<false>(idx, T, k, E, peer_L, R, 0, expert_count, expert_offset,
                                 rank_count, rank_offset, pos, row_src, workspace, status, stream);
}

}  // namespace moe
