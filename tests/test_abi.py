"""The C ABI without a GPU: exported symbols and host-side argument checks.

Every call here is rejected by validation before anything touches the GPU,
so the tests run on the CPU.
"""
import ctypes
import os
import re

import pytest

from paper_2607_26444_amd import moe

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "moe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(moe_\w+)\s*\(", text,
                                 flags=re.M)))


def test_header_declares_the_operator():
    names = declared_functions()
    for f in ("moe_layout", "moe_dispatch", "moe_combine", "moe_layout_workspace_bytes"):
        assert f in names


def test_library_exports_every_declared_symbol():
    lib = moe.lib()
    missing = [f for f in declared_functions() if not hasattr(lib, f)]
    assert not missing, missing


def test_binding_covers_every_declared_symbol():
    assert sorted(moe.EXPORTS) == declared_functions()


def test_binding_constants_match_the_header():
    text = open(HEADER).read()
    defines = dict(re.findall(r"^#define\s+(MOE_\w+)\s+\(?(-?\d+)u?\)?", text, flags=re.M))
    for name in ("MOE_PLAN_PARTS", "MOE_POLICY_STATIC", "MOE_EINVAL", "MOE_STATUS_CAPACITY"):
        assert name in defines, name
    assert moe.moe_version() == int(defines.pop("MOE_VERSION"))
    for name, value in defines.items():
        assert hasattr(moe, name), name
        assert getattr(moe, name) == int(value), name


def test_version_and_strerror():
    assert moe.moe_version() == 5
    for code in (0, -1, -2, -3, -4, -99):
        assert isinstance(moe.lib().moe_strerror(code), bytes)


@pytest.mark.parametrize("T,k,E,R,code", [
    (-1, 8, 256, 64, moe.MOE_EINVAL),       # negative tokens
    (16, 0, 256, 64, moe.MOE_EINVAL),       # k < 1
    (16, 33, 256, 64, moe.MOE_EINVAL),      # k > MOE_MAX_K
    (16, 8, 4, 2, moe.MOE_EINVAL),          # k > E
    (16, 8, 256, 60, moe.MOE_EINVAL),       # E % R != 0
    (16, 8, 2048, 64, moe.MOE_EINVAL),      # E > MOE_MAX_EXPERTS
    (2 ** 30, 8, 256, 64, moe.MOE_EINVAL),  # T*k beyond int32
])
def test_workspace_query_rejects_bad_shapes(T, k, E, R, code):
    out = ctypes.c_size_t(0)
    assert moe.lib().moe_layout_workspace_bytes(T, k, E, R, ctypes.byref(out)) == code


def test_workspace_size_covers_plan_and_counts():
    assert moe.moe_layout_workspace_bytes(16384, 8, 256, 64) >= (moe.MOE_PLAN_PARTS + 1) * 4
    assert moe.moe_layout_workspace_bytes(0, 8, 256, 64) >= (moe.MOE_PLAN_PARTS + 1) * 4
    assert moe.lib().moe_layout_workspace_bytes(16, 8, 256, 64, None) == moe.MOE_EINVAL


FAKE = ctypes.c_void_p(0x10000)      # never dereferenced: calls fail validation
MIS = ctypes.c_void_p(0x10008)       # 8-byte aligned, not 16
WS = ctypes.c_void_p(0x100000)       # 256-byte aligned "workspace"


def test_layout_argument_errors():
    L = moe.lib()
    n = moe.moe_layout_workspace_bytes(64, 8, 256, 64)
    ok = [FAKE, 64, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, WS, n, FAKE, None]
    bad = list(ok); bad[5] = None                      # null expert_count
    assert L.moe_layout(*bad) == moe.MOE_EINVAL
    bad = list(ok); bad[11] = ctypes.c_void_p(0x100010)  # misaligned workspace
    assert L.moe_layout(*bad) == moe.MOE_EWORKSPACE
    bad = list(ok); bad[12] = n - 4                    # workspace too small
    assert L.moe_layout(*bad) == moe.MOE_EWORKSPACE
    bad = list(ok); bad[4] = 48                        # E % R
    assert L.moe_layout(*bad) == moe.MOE_EINVAL


def _dispatch_args(**kw):
    n = moe.moe_layout_workspace_bytes(64, 8, 256, 64)
    a = dict(x=FAKE, xs=None, dtype=0, T=64, H=7168, k=8, E=256, R=64, idx=FAKE, pos=FAKE,
             ro=FAKE, rs=FAKE, rx=FAKE, rsc=None, pitch=0, cap=FAKE, ws=WS, wsb=n,
             st=FAKE, policy=0, waves=0, trace=None, tw=0, stream=None)
    a.update(kw)
    return list(a.values())


def test_dispatch_argument_errors():
    L = moe.lib()
    assert L.moe_dispatch_ex(*_dispatch_args(dtype=7)) == moe.MOE_EINVAL
    assert L.moe_dispatch_ex(*_dispatch_args(policy=5)) == moe.MOE_EINVAL
    assert L.moe_dispatch_ex(*_dispatch_args(policy=1, rs=None)) == moe.MOE_EINVAL
    assert L.moe_dispatch_ex(*_dispatch_args(x=MIS)) == moe.MOE_EALIGN
    assert L.moe_dispatch_ex(*_dispatch_args(H=7164)) == moe.MOE_EALIGN      # 2H % 16
    assert L.moe_dispatch_ex(*_dispatch_args(dtype=1, xs=FAKE, rsc=FAKE,
                                             H=7168 + 64)) == moe.MOE_EALIGN  # H % 128
    assert L.moe_dispatch_ex(*_dispatch_args(dtype=1, xs=None, rsc=FAKE)) == moe.MOE_EINVAL
    assert L.moe_dispatch_ex(*_dispatch_args(dtype=1, xs=FAKE, rsc=FAKE,
                                             pitch=64)) == moe.MOE_EINVAL     # < 224 B
    assert L.moe_dispatch_ex(*_dispatch_args(dtype=1, xs=FAKE, rsc=FAKE,
                                             pitch=226)) == moe.MOE_EALIGN
    assert L.moe_dispatch_ex(*_dispatch_args(wsb=16)) == moe.MOE_EWORKSPACE
    assert L.moe_dispatch_ex(*_dispatch_args(rx=None)) == moe.MOE_EINVAL
    assert L.moe_dispatch_ex(*_dispatch_args(trace=FAKE, tw=-1)) == moe.MOE_EINVAL
    for w in (-4, 2, 6, 20, 12292, 24576):             # not a divisor of the plan / of 4
        assert L.moe_dispatch_ex(*_dispatch_args(waves=w)) == moe.MOE_EINVAL
    assert L.moe_dispatch_ex(*_dispatch_args(policy=2, rs=FAKE, waves=96)) == moe.MOE_EINVAL
    # rows of 2 GiB or more: in-row offsets are 32-bit
    assert L.moe_dispatch_ex(*_dispatch_args(H=2 ** 30)) == moe.MOE_EINVAL


def test_combine_argument_errors():
    L = moe.lib()
    n = moe.moe_layout_workspace_bytes(64, 8, 256, 64)
    ok = [FAKE, FAKE, 64, 7168, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, WS, n, FAKE, 0, 0,
          None, 0, None]
    bad = list(ok); bad[11] = MIS                      # y misaligned
    assert L.moe_combine_ex(*bad) == moe.MOE_EALIGN
    bad = list(ok); bad[0] = None                      # null expert table
    assert L.moe_combine_ex(*bad) == moe.MOE_EINVAL
    bad = list(ok); bad[13] = 8
    assert L.moe_combine_ex(*bad) == moe.MOE_EWORKSPACE
    bad = list(ok); bad[4] = 300                       # k > MOE_MAX_K
    assert L.moe_combine_ex(*bad) == moe.MOE_EINVAL
    bad = list(ok); bad[15] = moe.MOE_POLICY_ROWS      # pull splits are dispatch-only
    assert L.moe_combine_ex(*bad) == moe.MOE_EINVAL
    bad = list(ok); bad[16] = 100                      # does not divide the plan
    assert L.moe_combine_ex(*bad) == moe.MOE_EINVAL
    bad = list(ok); bad[3] = 2 ** 30                   # a 2 GiB output row
    assert L.moe_combine_ex(*bad) == moe.MOE_EINVAL


def test_no_fallback_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(moe, "_lib", None)
    monkeypatch.setattr(moe, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        moe.lib()


def test_dedup_argument_errors():
    L = moe.lib()
    n = moe.moe_layout_dedup_workspace_bytes(64, 8, 256, 64)
    n_slot = moe.moe_layout_workspace_bytes(64, 8, 256, 64)
    assert n >= (moe.MOE_PLAN_PARTS + 1) * 4 + (2 * 64 + 1) * 4
    out = ctypes.c_size_t(0)
    assert L.moe_layout_dedup_workspace_bytes(16, 8, 256, 60, ctypes.byref(out)) == moe.MOE_EINVAL
    # layout
    ok = [FAKE, 64, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, WS, n, FAKE, None]
    assert L.moe_layout_dedup(*ok[:10], n - 4, *ok[11:]) == moe.MOE_EWORKSPACE
    bad = list(ok); bad[5] = None
    assert L.moe_layout_dedup(*bad) == moe.MOE_EINVAL
    bad = list(ok); bad[9] = ctypes.c_void_p(0x100010)
    assert L.moe_layout_dedup(*bad) == moe.MOE_EWORKSPACE
    # dispatch of pair rows: the pair-row workspace size is required
    d = [FAKE, None, 0, 64, 7168, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, None, 0, FAKE, WS, n,
         FAKE, None]
    bad = list(d); bad[16] = min(n, n_slot) - 4
    assert L.moe_dispatch_dedup(*bad) == moe.MOE_EWORKSPACE
    bad = list(d); bad[0] = MIS
    assert L.moe_dispatch_dedup(*bad) == moe.MOE_EALIGN
    bad = list(d); bad[2] = 5
    assert L.moe_dispatch_dedup(*bad) == moe.MOE_EINVAL
    # expand
    e = [FAKE, None, 0, 64, 7168, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0,
         FAKE, WS, n_slot, FAKE, None]
    bad = list(e); bad[13] = None                      # dedup_cap
    assert L.moe_expand(*bad) == moe.MOE_EINVAL
    bad = list(e); bad[2] = 1                          # fp8 without scale regions
    assert L.moe_expand(*bad) == moe.MOE_EINVAL
    bad = list(e); bad[4] = 7164
    assert L.moe_expand(*bad) == moe.MOE_EALIGN
    bad = list(e); bad[19] = 8
    assert L.moe_expand(*bad) == moe.MOE_EWORKSPACE
    # partial combine
    c = [FAKE, FAKE, 64, 7168, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, WS,
         n_slot, FAKE, None]
    bad = list(c); bad[14] = None                      # partial table
    assert L.moe_combine_local(*bad) == moe.MOE_EINVAL
    bad = list(c); bad[1] = None                       # weights
    assert L.moe_combine_local(*bad) == moe.MOE_EINVAL
    bad = list(c); bad[16] = 16
    assert L.moe_combine_local(*bad) == moe.MOE_EWORKSPACE
    # source-side sum
    s = [FAKE, 64, 7168, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, WS, n, FAKE, None]
    bad = list(s); bad[10] = MIS                       # y
    assert L.moe_combine_dedup(*bad) == moe.MOE_EALIGN
    bad = list(s); bad[12] = n - 4
    assert L.moe_combine_dedup(*bad) == moe.MOE_EWORKSPACE
    bad = list(s); bad[0] = None
    assert L.moe_combine_dedup(*bad) == moe.MOE_EINVAL


def test_layout_scratch_argument_errors():
    """moe_layout_scratch rejects bad arguments before any HIP call."""
    L = moe.lib()
    ws, nb = ctypes.c_void_p(), ctypes.c_size_t()
    ok = [FAKE, 64, 8, 256, 64, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
          ctypes.byref(ws), ctypes.byref(nb), None]
    for i, v in ((12, None), (13, None), (5, None), (11, None), (9, None), (3, 48), (1, -1),
                 (2, 33)):
        bad = list(ok)
        bad[i] = v
        assert L.moe_layout_scratch(*bad) == moe.MOE_EINVAL, i


def test_layout_scratch_array_covers_every_shape():
    """The library's workspace array (576 KiB) holds the workspace of every
    accepted shape: the count matrix is largest for E = 1 at the largest T."""
    sizes = [moe.moe_layout_workspace_bytes(2 ** 31 - 1, 1, E, 1) for E in range(1, 1025)]
    assert max(sizes) == 581888 == sizes[0]
    assert max(sizes) <= 576 * 1024
    for T in (0, 1, 255, 256, 257, 4096, 16384, 2 ** 20):
        for E in (1, 3, 16, 256, 1024):
            assert moe.moe_layout_workspace_bytes(T, 1, E, 1) <= 576 * 1024


_C_CLIENT = r"""
#include <stdio.h>
#include <string.h>
#include "moe.h"

int main(void) {
  size_t bytes = 0;
  if (moe_version() != MOE_VERSION) return 1;
  if (strcmp(moe_strerror(MOE_OK), "ok") != 0) return 2;
  if (moe_layout_workspace_bytes(16384, 8, 256, 64, &bytes) != MOE_OK) return 3;
  if (bytes < (size_t)(MOE_PLAN_PARTS + 1) * 4) return 4;
  if (moe_layout_workspace_bytes(16, 0, 256, 64, &bytes) != MOE_EINVAL) return 5;
  printf("%zu\n", bytes);
  return 0;
}
"""


def test_header_builds_a_c_program_that_links_the_library(tmp_path):
    """include/moe.h is a plain C header: a C99 program that includes it
    builds with every warning as an error, links libmoe.so and calls its
    host-side entry points (version, error text, workspace query)."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    moe.lib()
    src = tmp_path / "client.c"
    src.write_text(_C_CLIENT)
    exe = tmp_path / "client"
    libdir = os.path.dirname(moe.LIB_PATH)
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-I",
                        os.path.join(ROOT, "include"), str(src), "-o", str(exe), "-L", libdir,
                        "-l:libmoe.so", "-Wl,-rpath," + libdir],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert run.returncode == 0, (run.returncode, run.stderr)
    assert int(run.stdout.strip()) == moe.moe_layout_workspace_bytes(16384, 8, 256, 64)
