// C ABI of libmoe (declared in include/moe.h): argument validation and
// kernel launches.  Nothing here allocates, frees or synchronizes.

#include <limits.h>

#include <map>
#include <mutex>
#include <utility>

#include "dedup.h"
#include "moe_internal.h"

namespace moe {

int resident_waves(const void* kernel, size_t lds_bytes) {
  static std::mutex mu;
  static std::map<std::pair<int, const void*>, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = -1;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find({dev, kernel});
  if (it != cache.end()) return it->second;
  int cus = 0, blocks = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, kBlock, lds_bytes) !=
          hipSuccess ||
      cus < 1 || blocks < 1) {
    cus = 256;
    blocks = 4;
  }
  int w = cus * blocks * kWavesPerBlock;
  if (w > MOE_PLAN_PARTS) w = MOE_PLAN_PARTS;
  while (w > kWavesPerBlock && (MOE_PLAN_PARTS % w != 0 || w % kWavesPerBlock != 0)) --w;
  cache[{dev, kernel}] = w;
  return w;
}

int copy_waves(const void* kernel, int64_t per_wave, int64_t target, int min_waves) {
  const int cap = resident_waves(kernel, 0);
  int hi = kWavesPerBlock;
  while (hi * 2 <= cap) hi *= 2;
  const int lo = hi < min_waves ? hi : min_waves;
  const double want = (double)target / (double)(per_wave > 0 ? per_wave : 1);
  int w = lo;
  while (w < hi && (double)w * 1.41421356 < want) w *= 2;
  return w;
}

}  // namespace moe

namespace {

thread_local int g_last_hip_error = 0;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// An explicit wavefront count must split the plan into whole parts and
// launch whole workgroups.
bool waves_ok(int waves) {
  if (waves == 0) return true;
  return waves >= moe::kWavesPerBlock && waves <= MOE_PLAN_PARTS &&
         waves % moe::kWavesPerBlock == 0 && MOE_PLAN_PARTS % waves == 0;
}

// Kernels address within a row with 32-bit offsets: rows stay below 2 GiB.
bool row_fits(int64_t row_bytes) { return row_bytes <= (int64_t)INT32_MAX; }

int shape_ok(int64_t T, int k, int E, int R) {
  if (T < 0 || k < 1 || k > MOE_MAX_K || E < 1 || E > MOE_MAX_EXPERTS || R < 1 || k > E ||
      E % R != 0)
    return MOE_EINVAL;
  if (T > 0 && T > (int64_t)INT32_MAX / k) return MOE_EINVAL;
  return MOE_OK;
}

int launched(hipError_t err) { return moe::hip_status(err); }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

}  // namespace

int moe::hip_status(hipError_t err) {
  if (err == hipSuccess) return MOE_OK;
  g_last_hip_error = (int)err;
  return MOE_ELAUNCH;
}

extern "C" {

int moe_version(void) { return MOE_VERSION; }

const char* moe_strerror(int code) {
  switch (code) {
    case MOE_OK: return "ok";
    case MOE_EINVAL: return "invalid argument (null pointer or unsupported shape)";
    case MOE_EALIGN: return "misaligned pointer or row size";
    case MOE_EWORKSPACE: return "workspace too small or misaligned";
    case MOE_ELAUNCH: return "HIP kernel launch failed";
    default: return "unknown error";
  }
}

int moe_last_hip_error(void) { return g_last_hip_error; }

int moe_wall_clock_khz(int* khz) {
  if (!khz) return MOE_EINVAL;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err == hipSuccess) err = hipDeviceGetAttribute(khz, hipDeviceAttributeWallClockRate, dev);
  return launched(err);
}

int moe_layout_workspace_bytes(int64_t T, int k, int E, int R, size_t* out_bytes) {
  if (!out_bytes) return MOE_EINVAL;
  const int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  *out_bytes = moe::layout_geom(T, E).total;
  return MOE_OK;
}

int moe_layout(const int32_t* topk_idx, int64_t T, int k, int E, int R, int32_t* expert_count,
               int32_t* expert_offset, int32_t* rank_count, int32_t* rank_offset, int32_t* pos,
               int32_t* row_src, void* workspace, size_t workspace_bytes, uint32_t* status,
               void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (!expert_count || !expert_offset || !rank_count || !rank_offset || !workspace || !status)
    return MOE_EINVAL;
  if (T > 0 && (!topk_idx || !pos || !row_src)) return MOE_EINVAL;
  if (!aligned(workspace, 256) || workspace_bytes < moe::layout_geom(T, E).total)
    return MOE_EWORKSPACE;
  return launched(moe::launch_layout(topk_idx, T, k, E, R, -1, expert_count, expert_offset,
                                     rank_count, rank_offset, pos, row_src, workspace, status,
                                     as_stream(stream)));
}

int moe_layout_fixed(const int32_t* topk_idx, int64_t T, int k, int E, int R, int capacity,
                     int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
                     int32_t* rank_offset, int32_t* pos, int32_t* row_src, void* workspace,
                     size_t workspace_bytes, uint32_t* status, void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (capacity < 0 || (int64_t)E * capacity > (int64_t)INT32_MAX) return MOE_EINVAL;
  if (!expert_count || !expert_offset || !rank_count || !rank_offset || !workspace || !status)
    return MOE_EINVAL;
  if (T > 0 && (!topk_idx || !pos)) return MOE_EINVAL;
  if (capacity > 0 && !row_src) return MOE_EINVAL;
  if (!aligned(workspace, 256) || workspace_bytes < moe::layout_geom(T, E).total)
    return MOE_EWORKSPACE;
  return launched(moe::launch_layout(topk_idx, T, k, E, R, capacity, expert_count,
                                     expert_offset, rank_count, rank_offset, pos, row_src,
                                     workspace, status, as_stream(stream)));
}

}  // extern "C"

namespace {

// Shared by moe_dispatch_ex and moe_dispatch_dedup: plan and work tickets at
// the front of a workspace of at least need_bytes.
int dispatch_common(const void* x, const float* x_scales, int dtype, int64_t T, int H, int k,
                    int E, int R, const int32_t* topk_idx, const int32_t* pos,
                    const int32_t* rank_offset, const int32_t* row_src, const uint64_t* recv_x,
                    const uint64_t* recv_scales, int scale_pitch, const int32_t* recv_cap,
                    const void* workspace, size_t workspace_bytes, size_t need_bytes,
                    size_t ticket_offset, uint32_t* status, int policy, int waves,
                    uint64_t* trace, int trace_waves, int rows_hint, void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (H < 1 || (dtype != MOE_DTYPE_BF16 && dtype != MOE_DTYPE_FP8_E4M3)) return MOE_EINVAL;
  const bool fp8 = dtype == MOE_DTYPE_FP8_E4M3;
  if (!recv_x || !recv_cap || !rank_offset || !workspace || !status) return MOE_EINVAL;
  if (fp8 && (!x_scales || !recv_scales)) return MOE_EINVAL;
  if (T > 0 && (!x || !topk_idx || !pos)) return MOE_EINVAL;
  if (policy != MOE_POLICY_BALANCED && policy != MOE_POLICY_ROWS &&
      policy != MOE_POLICY_BY_RANK && policy != MOE_POLICY_DYNAMIC &&
      policy != MOE_POLICY_STATIC)
    return MOE_EINVAL;
  const bool pull = policy == MOE_POLICY_ROWS || policy == MOE_POLICY_BY_RANK;
  if (pull && T > 0 && !row_src) return MOE_EINVAL;
  if (!waves_ok(waves) || (waves && policy == MOE_POLICY_BY_RANK && waves % R != 0))
    return MOE_EINVAL;
  if (trace && trace_waves < 0) return MOE_EINVAL;
  const int64_t row_bytes = fp8 ? (int64_t)H : 2 * (int64_t)H;
  if (!row_fits(row_bytes)) return MOE_EINVAL;
  if (row_bytes % 16 != 0 || (fp8 && H % MOE_FP8_BLOCK != 0)) return MOE_EALIGN;
  if (!aligned(x, 16) || (fp8 && !aligned(x_scales, 4))) return MOE_EALIGN;
  const int scale_row = fp8 ? (H / MOE_FP8_BLOCK) * 4 : 0;
  const int pitch = (fp8 && scale_pitch == 0) ? scale_row : scale_pitch;
  if (fp8 && (pitch < scale_row)) return MOE_EINVAL;
  if (fp8 && pitch % 4 != 0) return MOE_EALIGN;
  if (!aligned(workspace, 256) || workspace_bytes < need_bytes) return MOE_EWORKSPACE;
  if (T == 0) return MOE_OK;
  moe::DispatchArgs a;
  a.x = static_cast<const uint8_t*>(x);
  a.x_scales = fp8 ? reinterpret_cast<const uint8_t*>(x_scales) : nullptr;
  a.tokens = T;
  a.row_bytes = row_bytes;
  a.scale_row_bytes = scale_row;
  a.scale_pitch = fp8 ? pitch : 0;
  a.k = k;
  a.L = E / R;
  a.topk_idx = topk_idx;
  a.pos = pos;
  a.rank_offset = rank_offset;
  a.recv_x = recv_x;
  a.recv_scales = fp8 ? recv_scales : nullptr;
  a.recv_cap = recv_cap;
  a.bound = static_cast<const int32_t*>(workspace);
  a.status = status;
  a.row_src = row_src;
  a.R = R;
  a.tickets = reinterpret_cast<uint32_t*>(static_cast<char*>(const_cast<void*>(workspace)) +
                                          ticket_offset);
  a.trace = trace;
  a.trace_waves = trace ? trace_waves : 0;
  a.launch_waves = waves;
  a.rows_hint = rows_hint;
  return launched(moe::launch_dispatch(a, policy, as_stream(stream)));
}

}  // namespace

extern "C" {

int moe_dispatch_ex(const void* x, const float* x_scales, int dtype, int64_t T, int H, int k,
                    int E, int R, const int32_t* topk_idx, const int32_t* pos,
                    const int32_t* rank_offset, const int32_t* row_src, const uint64_t* recv_x,
                    const uint64_t* recv_scales, int scale_pitch, const int32_t* recv_cap,
                    const void* workspace, size_t workspace_bytes, uint32_t* status,
                    int policy, int waves, uint64_t* trace, int trace_waves,
                    void* stream) {
  if (shape_ok(T, k, E, R)) return MOE_EINVAL;
  const moe::LayoutGeom g = moe::layout_geom(T, E);
  return dispatch_common(x, x_scales, dtype, T, H, k, E, R, topk_idx, pos, rank_offset, row_src,
                         recv_x, recv_scales, scale_pitch, recv_cap, workspace, workspace_bytes,
                         g.total, g.ticket_offset, status, policy, waves, trace, trace_waves,
                         0, stream);
}

int moe_dispatch(const void* x, const float* x_scales, int dtype, int64_t T, int H, int k, int E,
                 int R, const int32_t* topk_idx, const int32_t* pos, const int32_t* rank_offset,
                 const uint64_t* recv_x, const uint64_t* recv_scales, int scale_pitch,
                 const int32_t* recv_cap, const void* workspace, size_t workspace_bytes,
                 uint32_t* status, void* stream) {
  return moe_dispatch_ex(x, x_scales, dtype, T, H, k, E, R, topk_idx, pos, rank_offset, nullptr,
                         recv_x, recv_scales, scale_pitch, recv_cap, workspace, workspace_bytes,
                         status, MOE_POLICY_BALANCED, 0, nullptr, 0, stream);
}

}  // extern "C"

namespace {

// Shared by moe_combine_ex and moe_combine_dedup (unit weights: topk_w null).
int combine_common(const uint64_t* expert_y, const float* topk_w, bool unit_weights, int64_t T,
                   int H, int k, int E, int R, const int32_t* topk_idx, const int32_t* pos,
                   const int32_t* rank_offset, const int32_t* recv_cap, uint16_t* y,
                   const void* workspace, size_t workspace_bytes, size_t need_bytes,
                   size_t ticket_offset, uint32_t* status, int policy, int waves,
                   uint64_t* trace, int trace_waves, int rows_hint, void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (H < 1 || !row_fits(2 * (int64_t)H)) return MOE_EINVAL;
  if (!expert_y || !recv_cap || !rank_offset || !workspace || !status) return MOE_EINVAL;
  if (T > 0 && ((!unit_weights && !topk_w) || !topk_idx || !pos || !y)) return MOE_EINVAL;
  if (policy != MOE_POLICY_BALANCED && policy != MOE_POLICY_DYNAMIC &&
      policy != MOE_POLICY_STATIC)
    return MOE_EINVAL;
  if (!waves_ok(waves)) return MOE_EINVAL;
  if (trace && trace_waves < 0) return MOE_EINVAL;
  if ((2 * (int64_t)H) % 16 != 0 || !aligned(y, 16)) return MOE_EALIGN;
  if (!aligned(workspace, 256) || workspace_bytes < need_bytes) return MOE_EWORKSPACE;
  if (T == 0) return MOE_OK;
  moe::CombineArgs a;
  a.R = R;
  a.expert_y = expert_y;
  a.topk_w = unit_weights ? nullptr : topk_w;
  a.tokens = T;
  a.row_bytes = 2 * (int64_t)H;
  a.k = k;
  a.L = E / R;
  a.topk_idx = topk_idx;
  a.pos = pos;
  a.rank_offset = rank_offset;
  a.recv_cap = recv_cap;
  a.y = y;
  a.bound = static_cast<const int32_t*>(workspace);
  a.status = status;
  a.trace = trace;
  a.trace_waves = trace ? trace_waves : 0;
  a.launch_waves = waves;
  a.rows_hint = rows_hint;
  a.tickets = reinterpret_cast<uint32_t*>(static_cast<char*>(const_cast<void*>(workspace)) +
                                          ticket_offset) + moe::kTicketGroupWords;
  return launched(moe::launch_combine(a, policy, as_stream(stream)));
}

}  // namespace

extern "C" {

int moe_combine_ex(const uint64_t* expert_y, const float* topk_w, int64_t T, int H, int k,
                   int E, int R, const int32_t* topk_idx, const int32_t* pos,
                   const int32_t* rank_offset, const int32_t* recv_cap, uint16_t* y,
                   const void* workspace, size_t workspace_bytes, uint32_t* status,
                   int policy, int waves, uint64_t* trace, int trace_waves,
                   void* stream) {
  if (shape_ok(T, k, E, R)) return MOE_EINVAL;
  const moe::LayoutGeom g = moe::layout_geom(T, E);
  return combine_common(expert_y, topk_w, false, T, H, k, E, R, topk_idx, pos, rank_offset,
                        recv_cap, y, workspace, workspace_bytes, g.total, g.ticket_offset,
                        status, policy, waves, trace, trace_waves, 0, stream);
}

int moe_combine(const uint64_t* expert_y, const float* topk_w, int64_t T, int H, int k, int E,
                int R, const int32_t* topk_idx, const int32_t* pos, const int32_t* rank_offset,
                const int32_t* recv_cap, uint16_t* y, const void* workspace,
                size_t workspace_bytes, uint32_t* status, void* stream) {
  return moe_combine_ex(expert_y, topk_w, T, H, k, E, R, topk_idx, pos, rank_offset, recv_cap, y,
                        workspace, workspace_bytes, status, MOE_POLICY_BALANCED, 0, nullptr, 0,
                        stream);
}

int moe_expert_scale(const uint64_t* recv_x, const uint64_t* recv_scales, int scale_pitch,
                     int dtype, int H, int E, int R, int identity,
                     const int32_t* expert_offset, const int32_t* rank_offset,
                     const int32_t* recv_cap, const uint64_t* out_y, int64_t max_rows,
                     void* stream) {
  if (H < 1 || !row_fits(2 * (int64_t)H) || E < 1 || E > MOE_MAX_EXPERTS || R < 1 ||
      E % R != 0 || max_rows < 0)
    return MOE_EINVAL;
  if (dtype != MOE_DTYPE_BF16 && dtype != MOE_DTYPE_FP8_E4M3) return MOE_EINVAL;
  const bool fp8 = dtype == MOE_DTYPE_FP8_E4M3;
  if (!recv_x || !expert_offset || !rank_offset || !recv_cap || !out_y) return MOE_EINVAL;
  if (fp8 && !recv_scales) return MOE_EINVAL;
  if (H % 8 != 0 || (fp8 && H % MOE_FP8_BLOCK != 0)) return MOE_EALIGN;
  const int scale_row = fp8 ? (H / MOE_FP8_BLOCK) * 4 : 0;
  const int pitch = (fp8 && scale_pitch == 0) ? scale_row : scale_pitch;
  if (fp8 && pitch < scale_row) return MOE_EINVAL;
  if (fp8 && pitch % 4 != 0) return MOE_EALIGN;
  if (max_rows == 0) return MOE_OK;
  moe::ExpertArgs a;
  a.recv_x = recv_x;
  a.recv_scales = fp8 ? recv_scales : nullptr;
  a.scale_pitch = fp8 ? pitch : 0;
  a.H = H;
  a.E = E;
  a.L = E / R;
  a.identity = identity;
  a.expert_offset = expert_offset;
  a.rank_offset = rank_offset;
  a.recv_cap = recv_cap;
  a.out_y = out_y;
  a.max_rows = max_rows;
  return launched(moe::launch_expert_scale(a, fp8, as_stream(stream)));
}

int moe_layout_dedup_workspace_bytes(int64_t T, int k, int E, int R, size_t* out_bytes) {
  if (!out_bytes) return MOE_EINVAL;
  const int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  *out_bytes = moe::dedup_geom(T, k, R).total;
  return MOE_OK;
}

int moe_layout_dedup(const int32_t* topk_idx, int64_t T, int k, int E, int R, int32_t* tok_count,
                     int32_t* tok_offset, int32_t* tok_pos, int32_t* tok_src, void* workspace,
                     size_t workspace_bytes, uint32_t* status, void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (!tok_count || !tok_offset || !workspace || !status) return MOE_EINVAL;
  if (T > 0 && (!topk_idx || !tok_pos || !tok_src)) return MOE_EINVAL;
  const moe::DedupGeom d = moe::dedup_geom(T, k, R);
  if (!aligned(workspace, 256) || workspace_bytes < d.total) return MOE_EWORKSPACE;
  int32_t* spare = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + d.spare_offset);
  // the layout pass over peers: one "expert" per peer, one peer per "rank",
  // the expert indices binned by peer as they are read
  return launched(moe::launch_layout(topk_idx, T, k, R, R, -1, tok_count, tok_offset, spare,
                                     spare + R, tok_pos, tok_src, workspace, status,
                                     as_stream(stream), E / R));
}

int moe_dispatch_dedup(const void* x, const float* x_scales, int dtype, int64_t T, int H, int k,
                       int E, int R, const int32_t* topk_idx, const int32_t* tok_pos,
                       const int32_t* tok_offset, const uint64_t* recv_x,
                       const uint64_t* recv_scales, int scale_pitch, const int32_t* recv_cap,
                       const void* workspace, size_t workspace_bytes, uint32_t* status,
                       void* stream) {
  if (shape_ok(T, k, E, R)) return MOE_EINVAL;
  const moe::DedupGeom d = moe::dedup_geom(T, k, R);
  return dispatch_common(x, x_scales, dtype, T, H, k, E, R, topk_idx, tok_pos, tok_offset,
                         nullptr, recv_x, recv_scales, scale_pitch, recv_cap, workspace,
                         workspace_bytes, d.total, d.g.ticket_offset, status,
                         MOE_POLICY_BALANCED, 0, nullptr, 0, (k + 1) / 2, stream);
}

int moe_expand(const uint64_t* dedup_x, const uint64_t* dedup_scales, int dtype, int64_t T,
               int H, int k, int E, int R, const int32_t* topk_idx, const int32_t* pos,
               const int32_t* rank_offset, const int32_t* tok_pos, const int32_t* tok_offset,
               const int32_t* dedup_cap, const uint64_t* recv_x, const uint64_t* recv_scales,
               int scale_pitch, const int32_t* recv_cap, const void* workspace,
               size_t workspace_bytes, uint32_t* status, void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (H < 1 || (dtype != MOE_DTYPE_BF16 && dtype != MOE_DTYPE_FP8_E4M3)) return MOE_EINVAL;
  const bool fp8 = dtype == MOE_DTYPE_FP8_E4M3;
  if (!dedup_x || !dedup_cap || !recv_x || !recv_cap || !rank_offset || !tok_offset ||
      !workspace || !status)
    return MOE_EINVAL;
  if (fp8 && (!dedup_scales || !recv_scales)) return MOE_EINVAL;
  if (T > 0 && (!topk_idx || !pos || !tok_pos)) return MOE_EINVAL;
  const int64_t row_bytes = fp8 ? (int64_t)H : 2 * (int64_t)H;
  if (!row_fits(row_bytes)) return MOE_EINVAL;
  if (row_bytes % 16 != 0 || (fp8 && H % MOE_FP8_BLOCK != 0)) return MOE_EALIGN;
  const int scale_row = fp8 ? (H / MOE_FP8_BLOCK) * 4 : 0;
  const int pitch = (fp8 && scale_pitch == 0) ? scale_row : scale_pitch;
  if (fp8 && pitch < scale_row) return MOE_EINVAL;
  if (fp8 && pitch % 4 != 0) return MOE_EALIGN;
  if (!aligned(workspace, 256) || workspace_bytes < moe::layout_geom(T, E).total)
    return MOE_EWORKSPACE;
  if (T == 0) return MOE_OK;
  moe::ExpandArgs a;
  a.dedup_x = dedup_x;
  a.dedup_scales = fp8 ? dedup_scales : nullptr;
  a.dedup_cap = dedup_cap;
  a.recv_x = recv_x;
  a.recv_scales = fp8 ? recv_scales : nullptr;
  a.recv_cap = recv_cap;
  a.tokens = T;
  a.row_bytes = row_bytes;
  a.scale_row_bytes = scale_row;
  a.scale_pitch = fp8 ? pitch : 0;
  a.k = k;
  a.L = E / R;
  a.topk_idx = topk_idx;
  a.pos = pos;
  a.rank_offset = rank_offset;
  a.tok_pos = tok_pos;
  a.tok_offset = tok_offset;
  a.bound = static_cast<const int32_t*>(workspace);
  a.tickets = reinterpret_cast<uint32_t*>(static_cast<char*>(const_cast<void*>(workspace)) +
                                          moe::layout_geom(T, E).ticket_offset) +
              2 * moe::kTicketGroupWords;
  a.status = status;
  a.R = R;
  return launched(moe::launch_expand(a, as_stream(stream)));
}

int moe_combine_local(const uint64_t* expert_y, const float* topk_w, int64_t T, int H, int k,
                      int E, int R, const int32_t* topk_idx, const int32_t* pos,
                      const int32_t* rank_offset, const int32_t* recv_cap,
                      const int32_t* tok_pos, const int32_t* tok_offset,
                      const int32_t* part_cap, const uint64_t* partial, const void* workspace,
                      size_t workspace_bytes, uint32_t* status, void* stream) {
  int rc = shape_ok(T, k, E, R);
  if (rc) return rc;
  if (H < 1 || !row_fits(2 * (int64_t)H)) return MOE_EINVAL;
  if (!expert_y || !recv_cap || !rank_offset || !tok_offset || !part_cap || !partial ||
      !workspace || !status)
    return MOE_EINVAL;
  if (T > 0 && (!topk_w || !topk_idx || !pos || !tok_pos)) return MOE_EINVAL;
  if ((2 * (int64_t)H) % 16 != 0) return MOE_EALIGN;
  if (!aligned(workspace, 256) || workspace_bytes < moe::layout_geom(T, E).total)
    return MOE_EWORKSPACE;
  if (T == 0) return MOE_OK;
  moe::LocalArgs a;
  a.expert_y = expert_y;
  a.topk_w = topk_w;
  a.recv_cap = recv_cap;
  a.partial = partial;
  a.part_cap = part_cap;
  a.row_bytes = 2 * (int64_t)H;
  a.k = k;
  a.L = E / R;
  a.topk_idx = topk_idx;
  a.pos = pos;
  a.rank_offset = rank_offset;
  a.tok_pos = tok_pos;
  a.tok_offset = tok_offset;
  a.bound = static_cast<const int32_t*>(workspace);
  a.status = status;
  a.tokens = T;
  a.R = R;
  return launched(moe::launch_combine_local(a, as_stream(stream)));
}

int moe_combine_dedup(const uint64_t* partial, int64_t T, int H, int k, int E, int R,
                      const int32_t* topk_idx, const int32_t* tok_pos,
                      const int32_t* tok_offset, const int32_t* part_cap, uint16_t* y,
                      const void* workspace, size_t workspace_bytes, uint32_t* status,
                      void* stream) {
  if (shape_ok(T, k, E, R)) return MOE_EINVAL;
  const moe::DedupGeom d = moe::dedup_geom(T, k, R);
  // Sized and split as if every slot were a pair (its parts then count as
  // large at prefill-sized batches and take the claimed split): on MI355X
  // 6% faster at prefill and 11% at fp8 than sizing for half the slots,
  // 2% slower at the large workload, the same at decode.
  return combine_common(partial, nullptr, true, T, H, k, E, R, topk_idx, tok_pos, tok_offset,
                        part_cap, y, workspace, workspace_bytes, d.total, d.g.ticket_offset,
                        status, MOE_POLICY_BALANCED, 0, nullptr, 0, moe::slot_width(k), stream);
}

}  // extern "C"
