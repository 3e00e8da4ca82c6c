// CPU oracle for the MoE dispatch/combine hot path.
//
// TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
// load this file's library; only the tests, the smoke check and the
// benchmark's CPU-baseline leg do.  It shares no code, header, helper or
// table with the HIP library: it is a plain, slow, single-threaded reading of
// what the operator computes, written to be checked by eye against the paper.
//
// Built with: g++ -O2 -ffp-contract=off -shared -fPIC (see oracle/build.py).
//
// Notation (paper, Appendix D "Hierarchical Workload Partitioning for MoE
// Dispatch/Combine"): each token t has k routed slots j with destination
// expert e = topk_idx[t,j]; experts are spread over R peers ("ranks"), expert
// e living on peer r = e / (E/R).  Token placement is the per-expert counts,
// their prefix-sum offsets and each routed token's token-local offset inside
// its expert window; expert windows of one peer are contiguous and form the
// peer window whose payload is B_p.
//
// Readings where the paper is silent (each is listed in the design notes):
//  * one routed row per (token, expert) pair, ordered by (expert, token);
//  * slot value -1 marks an unused slot; an index outside [-1, E) and a
//    repeat of an expert already chosen earlier in the same row are treated
//    as unused and flagged in the status word (bits 1 and 2);
//  * combine is the top-k-weighted sum of a token's expert outputs (the
//    reduction of Section 6.1's reduction-bearing operators applied to the
//    routed rows), evaluated here in double precision and rounded once to
//    bf16 with round-to-nearest-even;
//  * rows whose region-local index reaches the region capacity are neither
//    written by dispatch nor read by combine, and set status bit 4.
//
// Parity pins for every function live in tests/test_oracle_*.py.

#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

namespace {

const uint32_t kBadIndex = 1u;   // index outside [-1, E)
const uint32_t kDupIndex = 2u;   // expert repeated within one token's row
const uint32_t kCapacity = 4u;   // region-local row >= region capacity

}  // namespace

extern "C" {

// ---------------------------------------------------------------------------
// Number formats.  Written from the IEEE-754 binary32 layout (bf16 is its
// upper 16 bits: 1 sign, 8 exponent, 7 fraction bits) and from the OCP 8-bit
// floating point specification (E4M3FN: bias 7, no infinities, S.1111.111 is
// NaN, largest finite 448).
// ---------------------------------------------------------------------------

double oracle_bf16_to_double(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return (double)f;
}

// Round a double to the nearest bf16 value, ties to even, in one step.
// bf16 keeps 8 significant bits and binary32's exponent range; below 2^-126
// its spacing is fixed at 2^-133 (subnormals).
uint16_t oracle_bf16_from_double(double x) {
  uint16_t sign = std::signbit(x) ? 0x8000u : 0u;
  if (std::isnan(x)) return (uint16_t)(sign | 0x7FC0u);
  if (std::isinf(x)) return (uint16_t)(sign | 0x7F80u);
  double ax = std::fabs(x);
  if (ax == 0.0) return sign;
  int e = std::ilogb(ax);                 // 2^e <= ax < 2^(e+1)
  int q = (e < -126 ? -126 : e) - 7;      // exponent of one unit in the last place
  double m = std::nearbyint(std::ldexp(ax, -q));  // exact scaling; ties-to-even
  double r = std::ldexp(m, q);
  if (r >= 0x1p128) return (uint16_t)(sign | 0x7F80u);  // overflow to infinity
  float f = (float)r;                     // exact: r has <= 8 significant bits
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return (uint16_t)(sign | (uint16_t)(u >> 16));
}

float oracle_fp8e4m3_to_float(uint8_t b) {
  int s = b >> 7, ex = (b >> 3) & 0xF, m = b & 7;
  if (ex == 15 && m == 7) return std::nanf("");
  double v = ex == 0 ? std::ldexp((double)m, -9)               // m/8 * 2^(1-7)
                     : std::ldexp(1.0 + m / 8.0, ex - 7);
  return (float)(s ? -v : v);
}

// ---------------------------------------------------------------------------
// Token placement (Appendix D, first and second level): per-expert and
// per-peer counts, exclusive prefix-sum offsets, and a stable position for
// every routed slot.  Plain counting sort keyed by expert, visiting tokens in
// order, so rows of one expert window are in token order.
//
// Outputs: expert_count[E], expert_offset[E+1], rank_count[R],
// rank_offset[R+1] (rank_offset[r] = expert_offset[r*E/R]), pos[T*k] (global
// row of each slot, -1 if unused), row_src[T*k] (slot t*k+j of each global
// row; -1 past the last row).  status |= bits.  Returns 0, or -1 on bad shape.
// ---------------------------------------------------------------------------
int oracle_layout(const int32_t* topk_idx, int64_t T, int32_t k, int32_t E,
                  int32_t R, int32_t* expert_count, int32_t* expert_offset,
                  int32_t* rank_count, int32_t* rank_offset, int32_t* pos,
                  int32_t* row_src, uint32_t* status) {
  if (T < 0 || k < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  const int64_t S = T * k;
  uint32_t st = 0;

  // Which slots are routed.
  std::vector<char> used((size_t)S, 0);
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t j = 0; j < k; ++j) {
      int32_t e = topk_idx[t * k + j];
      if (e == -1) continue;
      if (e < -1 || e >= E) { st |= kBadIndex; continue; }
      bool repeat = false;
      for (int32_t jj = 0; jj < j; ++jj)
        if (topk_idx[t * k + jj] == e) repeat = true;
      if (repeat) { st |= kDupIndex; continue; }
      used[(size_t)(t * k + j)] = 1;
    }
  }

  // Histogram over experts, then over peers.
  for (int32_t e = 0; e < E; ++e) expert_count[e] = 0;
  for (int64_t s = 0; s < S; ++s)
    if (used[(size_t)s]) expert_count[topk_idx[s]] += 1;
  for (int32_t r = 0; r < R; ++r) {
    rank_count[r] = 0;
    for (int32_t e = r * L; e < (r + 1) * L; ++e) rank_count[r] += expert_count[e];
  }

  // Exclusive prefix sums.
  expert_offset[0] = 0;
  for (int32_t e = 0; e < E; ++e) expert_offset[e + 1] = expert_offset[e] + expert_count[e];
  for (int32_t r = 0; r < R; ++r) rank_offset[r] = expert_offset[r * L];
  rank_offset[R] = expert_offset[E];

  // Token-local offsets: the next free row of each expert window.
  std::vector<int32_t> next(expert_offset, expert_offset + E);
  for (int64_t s = 0; s < S; ++s) row_src[s] = -1;
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t j = 0; j < k; ++j) {
      int64_t s = t * k + j;
      if (!used[(size_t)s]) { pos[s] = -1; continue; }
      int32_t p = next[topk_idx[s]]++;
      pos[s] = p;
      row_src[p] = (int32_t)s;
    }
  }
  *status |= st;
  return 0;
}

// ---------------------------------------------------------------------------
// Fixed-capacity placement (the low-latency form of the operator, Table 2's
// LL rows; the paper does not define the mode, this is the reading taken):
// every expert owns a window of C rows, expert e's window starting at e*C,
// so offsets are known without counting and receive regions (L*C rows per
// rank) can be sized before routing is known.  Within a window rows are in
// token order; a routed slot whose rank within its expert reaches C is
// dropped (pos = -1, status bit 4).  expert_count / rank_count count placed
// rows; expert_offset[e] = e*C, rank_offset[r] = r*L*C; row_src has E*C
// entries, -1 for rows no slot fills.
// ---------------------------------------------------------------------------
int oracle_layout_fixed(const int32_t* topk_idx, int64_t T, int32_t k, int32_t E, int32_t R,
                        int32_t C, int32_t* expert_count, int32_t* expert_offset,
                        int32_t* rank_count, int32_t* rank_offset, int32_t* pos,
                        int32_t* row_src, uint32_t* status) {
  if (T < 0 || k < 1 || E < 1 || R < 1 || E % R != 0 || C < 0) return -1;
  const int32_t L = E / R;
  uint32_t st = 0;
  for (int32_t e = 0; e < E; ++e) expert_count[e] = 0;
  for (int64_t i = 0; i < (int64_t)E * C; ++i) row_src[i] = -1;
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t j = 0; j < k; ++j) {
      const int64_t s = t * k + j;
      const int32_t e = topk_idx[s];
      pos[s] = -1;
      if (e == -1) continue;
      if (e < -1 || e >= E) { st |= kBadIndex; continue; }
      bool repeat = false;
      for (int32_t jj = 0; jj < j; ++jj)
        if (topk_idx[t * k + jj] == e) repeat = true;
      if (repeat) { st |= kDupIndex; continue; }
      if (expert_count[e] >= C) { st |= kCapacity; continue; }
      const int32_t p = e * C + expert_count[e];
      expert_count[e] += 1;
      pos[s] = p;
      row_src[p] = (int32_t)s;
    }
  }
  for (int32_t e = 0; e <= E; ++e) expert_offset[e] = e * C;
  for (int32_t r = 0; r < R; ++r) {
    rank_count[r] = 0;
    for (int32_t e = r * L; e < (r + 1) * L; ++e) rank_count[r] += expert_count[e];
    rank_offset[r] = r * L * C;
  }
  rank_offset[R] = E * C;
  *status |= st;
  return 0;
}

// ---------------------------------------------------------------------------
// Byte-balanced partition of the token range over P parts (Section 6.2 with a
// single memory tier: every unit has the same cost model, the fan-out cap
// does not bind, and a balanced split of the payload is what the list
// scheduler reaches).  The cost of token t is 1 + (number of its routed
// slots): one row read plus one row written per slot in dispatch, and the
// mirror image in combine.  With a(t) the cost of tokens before t and A the
// total, part p starts at bound[p] = the first t in [0, T] with
// a(t) * P >= p * A, so part p holds the tokens whose cost prefix lies in
// [p*A/P, (p+1)*A/P).  Output bound[P+1].
// ---------------------------------------------------------------------------
int oracle_plan(const int32_t* pos, int64_t T, int32_t k, int32_t P,
                int32_t* bound) {
  if (T < 0 || k < 1 || P < 1) return -1;
  std::vector<int64_t> a((size_t)T + 1, 0);
  for (int64_t t = 0; t < T; ++t) {
    int64_t c = 1;
    for (int32_t j = 0; j < k; ++j) c += pos[t * k + j] >= 0 ? 1 : 0;
    a[(size_t)t + 1] = a[(size_t)t] + c;
  }
  const int64_t A = a[(size_t)T];
  int64_t t = 0;
  for (int64_t p = 0; p <= P; ++p) {
    while (t < T && a[(size_t)t] * P < p * A) ++t;
    bound[p] = (int32_t)t;
  }
  return 0;
}

// ---------------------------------------------------------------------------
// Dispatch (Section 6.1 remote-slice transfers, one per routed slot: source
// row t of x, destination peer r, destination row pos - rank_offset[r] of
// that peer's receive region).  A pure byte copy of the row and, for fp8
// payloads, of its row of block scales; scale rows sit scale_pitch bytes
// apart and the bytes of a pitch past the scales are set to zero.
// recv_x[r] / recv_s[r] are host pointers to region r; recv_cap[r] is its
// capacity in rows.
// ---------------------------------------------------------------------------
int oracle_dispatch(const uint8_t* x, int64_t row_bytes, const uint8_t* x_scales,
                    int64_t scale_row_bytes, int64_t scale_pitch, int64_t T, int32_t k, int32_t E,
                    int32_t R, const int32_t* topk_idx, const int32_t* pos,
                    const int32_t* rank_offset, uint8_t* const* recv_x,
                    uint8_t* const* recv_s, const int32_t* recv_cap,
                    uint32_t* status) {
  if (T < 0 || k < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  uint32_t st = 0;
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t j = 0; j < k; ++j) {
      int32_t p = pos[t * k + j];
      if (p < 0) continue;
      int32_t r = topk_idx[t * k + j] / L;
      int64_t local = (int64_t)p - rank_offset[r];
      if (local >= recv_cap[r]) { st |= kCapacity; continue; }
      std::memcpy(recv_x[r] + local * row_bytes, x + t * row_bytes, (size_t)row_bytes);
      if (x_scales) {
        uint8_t* srow = recv_s[r] + local * scale_pitch;
        std::memcpy(srow, x_scales + t * scale_row_bytes, (size_t)scale_row_bytes);
        for (int64_t b = scale_row_bytes; b < scale_pitch; ++b) srow[b] = 0;
      }
    }
  }
  *status |= st;
  return 0;
}

// ---------------------------------------------------------------------------
// Stand-in expert used between dispatch and combine by the tests: expert e
// multiplies its rows by s_e = 1 + 0.01*e (or 1 for the identity expert).
// Computed in binary32 exactly as written -- s_e = 1.0f + (0.01f * e), bf16
// input: v * s_e; fp8 input: (q * block_scale) * s_e, one rounding per
// operation, no fused multiply-add -- then rounded to bf16 (nearest, ties to
// even).  Region r holds rows of experts r*L .. r*L+L-1 in expert order;
// expert_offset / rank_offset come from oracle_layout.
// ---------------------------------------------------------------------------
int oracle_expert_scale(uint8_t* const* recv_x, uint8_t* const* recv_s, int64_t scale_pitch,
                        int32_t payload_fp8, int32_t H, int32_t E, int32_t R,
                        int32_t identity, const int32_t* expert_offset,
                        const int32_t* rank_offset, const int32_t* recv_cap,
                        uint16_t* const* out) {
  if (H < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  for (int32_t e = 0; e < E; ++e) {
    const int32_t r = e / L;
    const float se = identity ? 1.0f : 1.0f + 0.01f * (float)e;
    for (int64_t g = expert_offset[e]; g < expert_offset[e + 1]; ++g) {
      int64_t local = g - rank_offset[r];
      if (local >= recv_cap[r]) continue;
      uint16_t* o = out[r] + local * H;
      for (int32_t h = 0; h < H; ++h) {
        float v;
        if (!payload_fp8) {
          const uint16_t* in = (const uint16_t*)recv_x[r] + local * H;
          v = (float)oracle_bf16_to_double(in[h]) * se;
        } else {
          const uint8_t* in = recv_x[r] + local * H;
          float sc;
          std::memcpy(&sc, recv_s[r] + local * scale_pitch + (h / 128) * 4, 4);
          float dq = oracle_fp8e4m3_to_float(in[h]) * sc;
          v = dq * se;
        }
        o[h] = oracle_bf16_from_double((double)v);
      }
    }
  }
  return 0;
}

// ---------------------------------------------------------------------------
// Combine: y[t] = sum over routed slots j of topk_w[t,j] * Y(row of slot j),
// where Y is the bf16 expert-output region of the slot's peer at the same
// region-local row dispatch wrote.  Sum in double, j ascending, then one
// rounding to bf16.  A token with no routed slot gets y = +0.
// ---------------------------------------------------------------------------
int oracle_combine(uint16_t* const* expert_y, const float* topk_w, int64_t T,
                   int32_t H, int32_t k, int32_t E, int32_t R,
                   const int32_t* topk_idx, const int32_t* pos,
                   const int32_t* rank_offset, const int32_t* recv_cap,
                   uint16_t* y, uint32_t* status) {
  if (T < 0 || H < 1 || k < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  uint32_t st = 0;
  std::vector<double> acc((size_t)H);
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t h = 0; h < H; ++h) acc[(size_t)h] = 0.0;
    for (int32_t j = 0; j < k; ++j) {
      int32_t p = pos[t * k + j];
      if (p < 0) continue;
      int32_t r = topk_idx[t * k + j] / L;
      int64_t local = (int64_t)p - rank_offset[r];
      if (local >= recv_cap[r]) { st |= kCapacity; continue; }
      const uint16_t* row = expert_y[r] + local * H;
      double w = (double)topk_w[t * k + j];
      for (int32_t h = 0; h < H; ++h) acc[(size_t)h] += w * oracle_bf16_to_double(row[h]);
    }
    for (int32_t h = 0; h < H; ++h) y[t * H + h] = oracle_bf16_from_double(acc[(size_t)h]);
  }
  *status |= st;
  return 0;
}

// ---------------------------------------------------------------------------
// Per-peer deduplicated placement (the peer windows of Appendix D, with each
// token sent once to every peer that hosts at least one of its experts --
// the reading taken for traffic that Section 6.2 calls uneven per peer).
// A token's routed slots (the same unused-slot rules as oracle_layout) are
// grouped by peer r = e / (E/R); the first slot of each group carries the
// group's row in peer window r, later slots of the group carry -1.  Rows of
// one peer window are in token order.
//
// Outputs: tok_count[R] (tokens sent to peer r), tok_offset[R+1] (exclusive
// prefix sums), tok_pos[T*k] (global row of the slot's (token, peer) pair on
// the group's first slot, -1 elsewhere), tok_src[T*k] (slot t*k+j of the
// first slot of each row, -1 past the last row).  status |= bits 1, 2.
// ---------------------------------------------------------------------------
int oracle_layout_dedup(const int32_t* topk_idx, int64_t T, int32_t k, int32_t E, int32_t R,
                        int32_t* tok_count, int32_t* tok_offset, int32_t* tok_pos,
                        int32_t* tok_src, uint32_t* status) {
  if (T < 0 || k < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  const int64_t S = T * k;
  uint32_t st = 0;
  // first[s]: slot s is routed and no earlier routed slot of its token has
  // an expert on the same peer
  std::vector<char> first((size_t)S, 0);
  for (int64_t t = 0; t < T; ++t) {
    std::vector<char> used((size_t)k, 0);
    for (int32_t j = 0; j < k; ++j) {
      const int32_t e = topk_idx[t * k + j];
      if (e == -1) continue;
      if (e < -1 || e >= E) { st |= kBadIndex; continue; }
      bool repeat = false;
      for (int32_t jj = 0; jj < j; ++jj)
        if (topk_idx[t * k + jj] == e) repeat = true;
      if (repeat) { st |= kDupIndex; continue; }
      used[(size_t)j] = 1;
      bool seen = false;
      for (int32_t jj = 0; jj < j; ++jj)
        if (used[(size_t)jj] && topk_idx[t * k + jj] / L == e / L) seen = true;
      first[(size_t)(t * k + j)] = seen ? 0 : 1;
    }
  }
  for (int32_t r = 0; r < R; ++r) tok_count[r] = 0;
  for (int64_t s = 0; s < S; ++s)
    if (first[(size_t)s]) tok_count[topk_idx[s] / L] += 1;
  tok_offset[0] = 0;
  for (int32_t r = 0; r < R; ++r) tok_offset[r + 1] = tok_offset[r] + tok_count[r];
  std::vector<int32_t> next(tok_offset, tok_offset + R);
  for (int64_t s = 0; s < S; ++s) tok_src[s] = -1;
  for (int64_t s = 0; s < S; ++s) {     // s = t*k + j ascending: token order
    if (!first[(size_t)s]) { tok_pos[s] = -1; continue; }
    const int32_t p = next[topk_idx[s] / L]++;
    tok_pos[s] = p;
    tok_src[p] = (int32_t)s;
  }
  *status |= st;
  return 0;
}

// Row of the (token, peer) pair of slot s = t*k + j in the deduplicated
// placement: tok_pos of the first slot of token t whose expert is on the same
// peer and that carries a row; -1 if there is none.
static int32_t pair_row(const int32_t* topk_idx, const int32_t* tok_pos, int64_t t, int32_t j,
                        int32_t k, int32_t L) {
  const int32_t r = topk_idx[t * k + j] / L;
  for (int32_t jj = 0; jj <= j; ++jj) {
    const int64_t s = t * k + jj;
    if (tok_pos[s] >= 0 && topk_idx[s] / L == r) return tok_pos[s];
  }
  return -1;
}

// ---------------------------------------------------------------------------
// Receiver-side expert permutation after a deduplicated dispatch: every
// routed slot (t, j) with expert e on peer r gets the row of its (token,
// peer) pair, copied from the deduplicated region r (row pair_row -
// tok_offset[r]) to the expert-ordered region r at row pos[t,j] -
// rank_offset[r] -- the same place a per-slot dispatch writes, so the result
// is that of oracle_dispatch.  fp8 scale rows are copied the same way, their
// pitch padding set to zero.  A source row at or past dedup_cap[r] or a
// destination row at or past recv_cap[r] is skipped and sets status bit 4.
// ---------------------------------------------------------------------------
int oracle_expand(uint8_t* const* dedup_x, uint8_t* const* dedup_s, int64_t row_bytes,
                  int64_t scale_row_bytes, int64_t scale_pitch, int64_t T, int32_t k, int32_t E,
                  int32_t R, const int32_t* topk_idx, const int32_t* pos,
                  const int32_t* rank_offset, const int32_t* tok_pos, const int32_t* tok_offset,
                  const int32_t* dedup_cap, uint8_t* const* recv_x, uint8_t* const* recv_s,
                  const int32_t* recv_cap, uint32_t* status) {
  if (T < 0 || k < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  uint32_t st = 0;
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t j = 0; j < k; ++j) {
      const int32_t p = pos[t * k + j];
      if (p < 0) continue;
      const int32_t r = topk_idx[t * k + j] / L;
      const int32_t q = pair_row(topk_idx, tok_pos, t, j, k, L);
      if (q < 0) continue;
      const int64_t src = (int64_t)q - tok_offset[r], dst = (int64_t)p - rank_offset[r];
      if (src >= dedup_cap[r] || dst >= recv_cap[r]) { st |= kCapacity; continue; }
      std::memcpy(recv_x[r] + dst * row_bytes, dedup_x[r] + src * row_bytes, (size_t)row_bytes);
      if (dedup_s) {
        uint8_t* srow = recv_s[r] + dst * scale_pitch;
        std::memcpy(srow, dedup_s[r] + src * scale_pitch, (size_t)scale_row_bytes);
        std::memset(srow + scale_row_bytes, 0, (size_t)(scale_pitch - scale_row_bytes));
      }
    }
  }
  *status |= st;
  return 0;
}

// ---------------------------------------------------------------------------
// Receiver-side partial combine after a deduplicated dispatch: for every
// (token, peer) pair, the top-k-weighted sum of the token's expert outputs on
// that peer, j ascending, in double, rounded once to bf16 and written to row
// pair_row - tok_offset[r] of the peer's partial region (the row that goes
// back to the token's source).  Expert-output rows are addressed as in
// oracle_combine.  The source then adds the partials of a token's peers
// (oracle_combine with unit weights over the pair rows).  Skipped rows set
// status bit 4: expert rows at or past recv_cap[r] (not summed) and pair
// rows at or past part_cap[r] (not written).
// ---------------------------------------------------------------------------
int oracle_combine_local(uint16_t* const* expert_y, const float* topk_w, int64_t T, int32_t H,
                         int32_t k, int32_t E, int32_t R, const int32_t* topk_idx,
                         const int32_t* pos, const int32_t* rank_offset,
                         const int32_t* recv_cap, const int32_t* tok_pos,
                         const int32_t* tok_offset, const int32_t* part_cap,
                         uint16_t* const* partial, uint32_t* status) {
  if (T < 0 || H < 1 || k < 1 || E < 1 || R < 1 || E % R != 0) return -1;
  const int32_t L = E / R;
  uint32_t st = 0;
  std::vector<double> acc((size_t)H);
  for (int64_t t = 0; t < T; ++t) {
    for (int32_t j0 = 0; j0 < k; ++j0) {
      const int32_t q = tok_pos[t * k + j0];
      if (q < 0) continue;                 // not the first slot of a pair
      const int32_t r = topk_idx[t * k + j0] / L;
      for (int32_t h = 0; h < H; ++h) acc[(size_t)h] = 0.0;
      for (int32_t j = j0; j < k; ++j) {
        const int32_t p = pos[t * k + j];
        if (p < 0 || topk_idx[t * k + j] / L != r) continue;
        const int64_t local = (int64_t)p - rank_offset[r];
        if (local >= recv_cap[r]) { st |= kCapacity; continue; }
        const uint16_t* row = expert_y[r] + local * H;
        const double w = (double)topk_w[t * k + j];
        for (int32_t h = 0; h < H; ++h) acc[(size_t)h] += w * oracle_bf16_to_double(row[h]);
      }
      const int64_t dst = (int64_t)q - tok_offset[r];
      if (dst >= part_cap[r]) { st |= kCapacity; continue; }
      uint16_t* o = partial[r] + dst * H;
      for (int32_t h = 0; h < H; ++h) o[h] = oracle_bf16_from_double(acc[(size_t)h]);
    }
  }
  *status |= st;
  return 0;
}

}  // extern "C"
