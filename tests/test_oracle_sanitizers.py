"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Every parity claim rests on the oracle, which indexes raw region tables,
pitches and offset arrays.  Here oracle/moe_oracle.cpp is built with
-fsanitize=address,undefined (no recovery: the first report aborts) into a
temporary directory and every pin runs against that build in a child
process, with the sanitizer runtime preloaded (the Python interpreter itself
is not instrumented).  Two planted mistakes -- a write one element past an
output array and an integer division by zero -- must each abort the child
with the sanitizer's report, which shows the instrumentation is live.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "moe_oracle.cpp")

FLAGS = ["-O1", "-g", "-std=c++17", "-ffp-contract=off", "-fno-omit-frame-pointer",
         "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
         "-shared", "-fPIC"]

RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
oracle.use_library({lib!r})
import oracle_pins as pins
for pin in pins.ALL_PINS:
    pin()
    print("PIN_OK", pin.__name__, flush=True)
print("ALL_PINS_PASSED", flush=True)
"""

# (name, original fragment, planted mistake, sanitizer report expected)
PLANTED = [
    ("rank_offset_overflow", "rank_offset[R] = expert_offset[E];",
     "rank_offset[R + 1] = expert_offset[E];", "heap-buffer-overflow"),
    ("division_by_zero", "const int32_t L = E / R;\n  const int64_t S = T * k;",
     "const int32_t L = E / (R - R);\n  const int64_t S = T * k;", "division by zero"),
]


def _asan_runtime():
    r = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        pytest.skip("no AddressSanitizer runtime for g++")
    return path


def _build(src_text, tmp, name):
    cpp = os.path.join(tmp, f"{name}.cpp")
    lib = os.path.join(tmp, f"lib{name}.so")
    with open(cpp, "w") as f:
        f.write(src_text)
    subprocess.run(["g++", *FLAGS, cpp, "-o", lib], check=True)
    return lib


def _run_pins(lib, asan):
    code = RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    env = dict(os.environ)
    # the sanitizer runtime must come first; anything already preloaded stays
    env["LD_PRELOAD"] = " ".join(p for p in (asan, os.environ.get("LD_PRELOAD", "")) if p)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["OMP_NUM_THREADS"] = "1"
    return subprocess.run([sys.executable, "-c", code], capture_output=True, text=True,
                          timeout=600, env=env)


def test_oracle_pins_pass_under_asan_and_ubsan():
    asan = _asan_runtime()
    with tempfile.TemporaryDirectory() as tmp:
        lib = _build(open(SRC).read(), tmp, "oracle_san")
        out = _run_pins(lib, asan)
    assert out.returncode == 0 and "ALL_PINS_PASSED" in out.stdout, \
        (out.returncode, out.stdout[-2000:], out.stderr[-4000:])


@pytest.mark.parametrize("name,before,after,report", PLANTED, ids=[p[0] for p in PLANTED])
def test_planted_fault_is_reported(name, before, after, report):
    asan = _asan_runtime()
    src = open(SRC).read()
    assert src.count(before) >= 1, f"{name}: fragment not found"
    with tempfile.TemporaryDirectory() as tmp:
        lib = _build(src.replace(before, after, 1), tmp, name)
        out = _run_pins(lib, asan)
    assert out.returncode != 0, out.stdout[-1000:]
    assert report in out.stderr, out.stderr[-3000:]
