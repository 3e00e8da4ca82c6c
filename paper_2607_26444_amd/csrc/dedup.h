// Internal declarations of the per-peer deduplicated path (dedup.hip):
// token placement with one row per (token, peer) pair, the receiver-side
// expansion of pair rows into expert order and the receiver-side partial
// combine.  Dispatch of pair rows and the source-side sum of partials reuse
// the dispatch and combine kernels.
#pragma once

#include "moe_internal.h"

namespace moe {

// Layout of the workspace of moe_layout_dedup: the layout pass over peers
// (plan first, as every copy kernel expects), then the two arrays the layout
// pass writes but the caller does not see.
struct DedupGeom {
  LayoutGeom g;          // layout_geom(T, R)
  size_t spare_offset;   // int32 [R] + int32 [R + 1]
  size_t total;
};

DedupGeom dedup_geom(int64_t T, int k, int R);

struct ExpandArgs {
  const uint64_t* dedup_x;       // [R] pair-row region bases
  const uint64_t* dedup_scales;  // [R] or nullptr
  const int32_t* dedup_cap;
  const uint64_t* recv_x;        // [R] expert-ordered region bases
  const uint64_t* recv_scales;
  const int32_t* recv_cap;
  int64_t tokens;                // T
  int64_t row_bytes;
  int32_t scale_row_bytes;
  int32_t scale_pitch;
  int32_t k;
  int32_t L;
  const int32_t* topk_idx;
  const int32_t* pos;
  const int32_t* rank_offset;
  const int32_t* tok_pos;
  const int32_t* tok_offset;
  const int32_t* bound;          // plan of the per-slot layout
  uint32_t* tickets;             // claimed parts: {next, done}, zeroed by the layout
  uint32_t* status;
  int32_t R;                     // ranks
};

hipError_t launch_expand(const ExpandArgs& a, hipStream_t stream);

struct LocalArgs {
  const uint64_t* expert_y;      // [R] bf16 expert-output region bases
  const float* topk_w;
  const int32_t* recv_cap;
  const uint64_t* partial;       // [R] bf16 partial region bases
  const int32_t* part_cap;
  int64_t row_bytes;             // 2H
  int32_t k;
  int32_t L;
  const int32_t* topk_idx;
  const int32_t* pos;
  const int32_t* rank_offset;
  const int32_t* tok_pos;
  const int32_t* tok_offset;
  const int32_t* bound;          // plan of the per-slot layout
  uint32_t* status;
  int64_t tokens;                // T
  int32_t R;                     // ranks
};

hipError_t launch_combine_local(const LocalArgs& a, hipStream_t stream);

}  // namespace moe
