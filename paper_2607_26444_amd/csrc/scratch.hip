// moe_layout_scratch: moe_layout into the library's own per-device
// workspace, for callers that cannot allocate device memory (code under
// graph capture, tight serving loops).
//
// The workspace of moe_layout (partition plan, work tickets, per-chunk count
// matrix) is bounded for every shape the library accepts: the count matrix
// has at most max(1, 32768 / E) rows of E rounded up to 4 int32, which is
// largest at E = 1 (512 KiB), so the whole workspace never exceeds
// 581888 bytes.  It lives in one file-scope device array per GPU.  Host code
// never passes that array's name to a kernel: the name is a host-side
// stand-in; its device address is looked up once per device with
// hipGetSymbolAddress and kept per device.

#include <mutex>

#include "moe_internal.h"

namespace {

constexpr size_t kScratchBytes = 576u << 10;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on the current device (looked up on the first
// call for that device, with that device current).
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

int moe_layout_scratch(const int32_t* topk_idx, int64_t T, int k, int E, int R,
                       int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
                       int32_t* rank_offset, int32_t* pos, int32_t* row_src, uint32_t* status,
                       void** workspace, size_t* workspace_bytes, void* stream) {
  // argument errors first: nothing below runs (no HIP call) on bad input
  if (!workspace || !workspace_bytes) return MOE_EINVAL;
  if (!expert_count || !expert_offset || !rank_count || !rank_offset || !status)
    return MOE_EINVAL;
  if (T > 0 && (!topk_idx || !pos || !row_src)) return MOE_EINVAL;
  size_t need = 0;
  int rc = moe_layout_workspace_bytes(T, k, E, R, &need);
  if (rc != MOE_OK) return rc;
  if (need > kScratchBytes) return MOE_EWORKSPACE;
  void* ws = nullptr;
  rc = moe::hip_status(scratch_address(&ws));
  if (rc != MOE_OK) return rc;
  rc = moe_layout(topk_idx, T, k, E, R, expert_count, expert_offset, rank_count, rank_offset,
                  pos, row_src, ws, kScratchBytes, status, stream);
  if (rc == MOE_OK) {
    *workspace = ws;
    *workspace_bytes = need;
  }
  return rc;
}

}  // extern "C"
