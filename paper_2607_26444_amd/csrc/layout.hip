// Token placement and partition plan (paper Appendix D, first to third
// level; Section 6.2 for the byte-balanced split).
//
// Two kernels, both one workgroup per chunk of tokens (a batch of at most
// 256 tokens needs only the second, which then counts for itself):
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
#pragma unroll
    for (int j = 0; j < KW; ++j)
      if (j < k) ev[j] = idx[t * k + j];
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

// Exclusive scan of one int64 per thread over the 256-thread block; also
// returns the block total.  `scratch` holds kWavesPerBlock int64.
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t v, int64_t* scratch,
                                                        int64_t& total) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
  int64_t inc = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int64_t o = __shfl_up(inc, d, kWave);
    if (lane >= d) inc += o;
  }
  if (lane == kWave - 1) scratch[w] = inc;
  __syncthreads();
  int64_t before = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    const int64_t s = scratch[i];
    before += (i < w) ? s : 0;
    total += s;
  }
  __syncthreads();
  return before + inc - v;
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

// SINGLE: the whole batch is one sub-chunk (T <= kBlock), so this kernel
// also does the counting (no layout_count launch): the totals are the
// popcounts of its own bitmaps.
// FIXED: fixed-capacity windows of C rows per expert (expert e's window
// starts at e*C); a slot whose rank within its expert reaches C is dropped.
template <int KW, bool SINGLE, bool FIXED>
__global__ __launch_bounds__(kBlock) void layout_place_kernel(
    const int32_t* __restrict__ idx, int64_t T, int k, int E, int peer_L, int R, int C,
    int64_t chunk_tokens, int nc, int ncp, const int32_t* __restrict__ counts, int32_t* __restrict__ expert_count,
    int32_t* __restrict__ expert_offset, int32_t* __restrict__ rank_count,
    int32_t* __restrict__ rank_offset, int32_t* __restrict__ pos,
    int32_t* __restrict__ row_src, int32_t* __restrict__ bound, uint32_t* __restrict__ tickets,
    uint32_t* __restrict__ status) {
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
  if (SINGLE) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < KW; ++j)
      if (ok0[j]) atomicOr(&mask[w * E + ev0[j]], 1ull << lane);
    __syncthreads();
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
    int32_t* part_t = woff;                   // [groups][ncp], free until placement
    int32_t* part_p = woff + groups * ncp;
    if (gi < groups) {
      int4 ta = {0, 0, 0, 0}, pa = {0, 0, 0, 0};
      for (int r0 = gi; r0 < nc; r0 += groups * kCountBatch) {
        int4 v[kCountBatch];
#pragma unroll
        for (int u = 0; u < kCountBatch; ++u) {
          const int r = min(r0 + u * groups, nc - 1);  // past nc: re-read, ignored
          v[u] = reinterpret_cast<const int4*>(counts + (int64_t)r * ncp)[li];
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
  // One scan for both sums: totals in the high 32 bits, this chunk's prefix
  // in the low 32 (all sums are below 2^31, so no carry crosses).
  int64_t packed_total = 0;
  const int64_t packed = block_exclusive_scan((my_tot << 32) | my_pre, scan, packed_total);
  int64_t run = packed >> 32;                      // rows before my experts
  const int64_t n_total = packed_total >> 32;       // placed rows N
  const int64_t pre_total = packed_total & 0xFFFFFFFFll;  // placed rows before chunk
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
    if (tid < 8) tickets[tid] = 0u;  // work tickets of dispatch, combine, expand
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
    if (!SINGLE) {
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
    int nplaced = 0;
#pragma unroll
    for (int j = 0; j < KW; ++j) {
      if (t < c1 && j < k) {
        int p = -1;
        if (ok[j]) {
          const int e = ev[j];
          const int r = woff[w * E + e] + __popcll(mask[w * E + e] & below);
          if (!FIXED || r - e * C < C) {
            p = r;
            row_src[p] = (int32_t)(t * k + j);
            ++nplaced;
          } else {
            st |= MOE_STATUS_CAPACITY;
          }
        }
        pos[t * k + j] = p;
      }
    }
    // Plan boundaries inside this sub-chunk: token t owns the parts p with
    // a_t*P < p*A <= (a_t + cost_t)*P, each starting at token t+1.  In cost
    // units, part p starts inside unit ceil(p*A/P) - 1, so the sub-chunk's
    // units are mapped to their tokens in LDS and the parts are written
    // part-major: lane l of each store takes part p0 + l (coalesced; a token
    // may own hundreds of parts when there are few tokens).
    const int64_t cost = (t < c1) ? 1 + nplaced : 0;
    int64_t sub_total = 0;
    const int64_t ex = block_exclusive_scan(cost, scan, sub_total);
    for (int64_t u = ex; u < ex + cost; ++u) owner[u] = (uint16_t)tid;
    __syncthreads();
    const int64_t p_first = (cost_base * P) / A + 1;
    const int64_t p_last = ((cost_base + sub_total) * P) / A;
    for (int64_t p = p_first + tid; p <= p_last; p += kBlock)
      bound[p] = (int32_t)(s0 + owner[(p * A - 1) / P - cost_base] + 1);
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

template <int KW, bool FIXED>
hipError_t launch_layout_kw(const int32_t* idx, int64_t T, int k, int E, int peer_L, int R, int C,
                            int32_t* expert_count, int32_t* expert_offset,
                            int32_t* rank_count, int32_t* rank_offset, int32_t* pos,
                            int32_t* row_src, void* workspace, uint32_t* status,
                            hipStream_t stream) {
  const LayoutGeom g = layout_geom(T, E);
  int32_t* bound = reinterpret_cast<int32_t*>(workspace);
  int32_t* counts = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + g.counts_offset);
  uint32_t* tickets = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + g.ticket_offset);
  const size_t lds_count = (size_t)kWavesPerBlock * E * 8 + (size_t)E * 4;
  // woff also holds the two [groups][ncp] count partials (groups * ncp <=
  // 4 * kBlock int32 each) before placement starts.
  const size_t woff_ints = (size_t)kWavesPerBlock * E > 8 * kBlock ? (size_t)kWavesPerBlock * E
                                                                    : 8 * kBlock;
  const size_t lds_place = (size_t)kWavesPerBlock * E * 8 + kWavesPerBlock * 8 +
                           (size_t)E * 4 + (size_t)(E + 1) * 4 + woff_ints * 4 +
                           (size_t)kBlock * (1 + KW) * 2;
  if (g.nc == 1 && T <= kBlock) {
    hipLaunchKernelGGL((layout_place_kernel<KW, true, FIXED>), dim3(1), dim3(kBlock), lds_place,
                       stream, idx, T, k, E, peer_L, R, C, g.chunk_tokens, g.nc, g.ncp, counts,
                       expert_count,
                       expert_offset, rank_count, rank_offset, pos, row_src, bound, tickets,
                       status);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(layout_count_kernel<KW>, dim3(g.nc), dim3(kBlock), lds_count, stream,
                     idx, T, k, E, peer_L, g.chunk_tokens, g.ncp, counts, status);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL((layout_place_kernel<KW, false, FIXED>), dim3(g.nc), dim3(kBlock),
                     lds_place, stream, idx, T, k, E, peer_L, R, C, g.chunk_tokens, g.nc, g.ncp, counts,
                     expert_count,
                     expert_offset, rank_count, rank_offset, pos, row_src, bound, tickets,
                     status);
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
  g.counts_offset = g.ticket_offset + 256;
  g.counts_bytes = (size_t)g.nc * g.ncp * 4;
  g.total = g.counts_offset + (g.counts_bytes + 255) / 256 * 256;
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
