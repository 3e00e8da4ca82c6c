"""The C ABI from a C program, without Python or PyTorch: a C99 client
allocates device memory with the HIP runtime, runs moe_layout, moe_dispatch
and moe_combine on a small batch and checks the result on the host against
a closed form: with every routing weight 1 and the dispatched rows used as
the expert outputs, y = bf16(k * x), exactly x * k for k a power of two."""
import os
import shutil
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_CLIENT = r"""
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <hip/hip_runtime_api.h>
#include "moe.h"

#define CHECK_HIP(x) do { if ((x) != hipSuccess) { printf("hip error line %d\n", __LINE__); return 10; } } while (0)
#define CHECK_MOE(x) do { int rc_ = (x); if (rc_ != MOE_OK) { printf("moe error %d line %d: %s\n", rc_, __LINE__, moe_strerror(rc_)); return 11; } } while (0)

static float bf16_to_float(uint16_t b) { uint32_t u = (uint32_t)b << 16; float f; memcpy(&f, &u, 4); return f; }

int main(void) {
  const int64_t T = 1000; const int H = 1024, E = 64, R = 8, k = 4;
  const size_t rb = 2 * (size_t)H, nslot = (size_t)T * k;
  int32_t* idx = malloc(nslot * 4); float* w = malloc(nslot * 4);
  uint16_t* x = malloc((size_t)T * H * 2); uint16_t* y = malloc((size_t)T * H * 2);
  for (int64_t t = 0; t < T; ++t)
    for (int j = 0; j < k; ++j) { idx[t * k + j] = (int32_t)((t * 7 + j * 13) % E); w[t * k + j] = 1.0f; }
  for (int64_t i = 0; i < T * H; ++i) {            /* bf16 of small multiples of 1/8 */
    float f = (float)((i * 37) % 61 - 30) * 0.125f; uint32_t u; memcpy(&u, &f, 4); x[i] = (uint16_t)(u >> 16);
  }
  size_t ws_bytes = 0;
  CHECK_MOE(moe_layout_workspace_bytes(T, k, E, R, &ws_bytes));
  void *d_idx, *d_w, *d_x, *d_y, *d_ws, *d_ec, *d_eo, *d_rc, *d_ro, *d_pos, *d_rs, *d_st;
  CHECK_HIP(hipMalloc(&d_idx, nslot * 4)); CHECK_HIP(hipMalloc(&d_w, nslot * 4));
  CHECK_HIP(hipMalloc(&d_x, (size_t)T * rb)); CHECK_HIP(hipMalloc(&d_y, (size_t)T * rb));
  CHECK_HIP(hipMalloc(&d_ws, ws_bytes)); CHECK_HIP(hipMalloc(&d_ec, E * 4));
  CHECK_HIP(hipMalloc(&d_eo, (E + 1) * 4)); CHECK_HIP(hipMalloc(&d_rc, R * 4));
  CHECK_HIP(hipMalloc(&d_ro, (R + 1) * 4)); CHECK_HIP(hipMalloc(&d_pos, nslot * 4));
  CHECK_HIP(hipMalloc(&d_rs, nslot * 4)); CHECK_HIP(hipMalloc(&d_st, 4));
  CHECK_HIP(hipMemcpy(d_idx, idx, nslot * 4, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_w, w, nslot * 4, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_x, x, (size_t)T * rb, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemset(d_st, 0, 4));
  CHECK_MOE(moe_layout(d_idx, T, k, E, R, d_ec, d_eo, d_rc, d_ro, d_pos, d_rs, d_ws, ws_bytes, d_st, NULL));
  int32_t rc[8];
  CHECK_HIP(hipMemcpy(rc, d_rc, R * 4, hipMemcpyDeviceToHost));
  /* receive regions: one allocation, regions at 4 KiB offsets */
  size_t off[8], total = 0;
  for (int r = 0; r < R; ++r) { off[r] = total; total += ((size_t)rc[r] * rb + 4095) / 4096 * 4096; }
  void *d_reg, *d_tab, *d_cap;
  CHECK_HIP(hipMalloc(&d_reg, total + 4096)); CHECK_HIP(hipMalloc(&d_tab, R * 8)); CHECK_HIP(hipMalloc(&d_cap, R * 4));
  uint64_t tab[8];
  for (int r = 0; r < R; ++r) tab[r] = (uint64_t)(uintptr_t)d_reg + off[r];
  CHECK_HIP(hipMemcpy(d_tab, tab, R * 8, hipMemcpyHostToDevice));
  CHECK_HIP(hipMemcpy(d_cap, rc, R * 4, hipMemcpyHostToDevice));
  CHECK_MOE(moe_dispatch(d_x, NULL, MOE_DTYPE_BF16, T, H, k, E, R, d_idx, d_pos, d_ro, d_tab, NULL, 0,
                         d_cap, d_ws, ws_bytes, d_st, NULL));
  CHECK_MOE(moe_combine(d_tab, d_w, T, H, k, E, R, d_idx, d_pos, d_ro, d_cap, d_y, d_ws, ws_bytes,
                        d_st, NULL));
  CHECK_HIP(hipDeviceSynchronize());
  uint32_t st = 0;
  CHECK_HIP(hipMemcpy(&st, d_st, 4, hipMemcpyDeviceToHost));
  CHECK_HIP(hipMemcpy(y, d_y, (size_t)T * rb, hipMemcpyDeviceToHost));
  if (st != 0) { printf("status %u\n", st); return 12; }
  for (int64_t i = 0; i < T * H; ++i)
    if (bf16_to_float(y[i]) != (float)k * bf16_to_float(x[i])) { printf("y mismatch at %lld\n", (long long)i); return 13; }
  int64_t n = 0;
  for (int r = 0; r < R; ++r) n += rc[r];
  printf("ok %lld rows\n", (long long)n);
  return 0;
}
"""


def test_c_program_runs_the_chain():
    from paper_2607_26444_amd import moe
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    moe.lib()
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "client.c")
        exe = os.path.join(d, "client")
        with open(src, "w") as f:
            f.write(_CLIENT)
        libdir = os.path.dirname(moe.LIB_PATH)
        rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
        r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                            "-I", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"),
                            src, "-o", exe, "-L", libdir, "-l:libmoe.so",
                            "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                            "-Wl,-rpath," + libdir, "-Wl,-rpath," + os.path.join(rocm, "lib")],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        run = subprocess.run([exe], capture_output=True, text=True, timeout=120)
        assert run.returncode == 0, (run.returncode, run.stdout, run.stderr)
        assert run.stdout.startswith("ok 4000 rows"), run.stdout
