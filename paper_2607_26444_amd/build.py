"""Build libmoe.so (HIP, gfx950) in-tree with hipcc.

python -m paper_2607_26444_amd.build [--isa DIR]

--isa DIR keeps the device assembly (*.s) of every source under DIR.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libmoe.so")
SOURCES = ["api.hip", "layout.hip", "dispatch.hip", "combine.hip", "expert.hip", "dedup.hip",
           "scratch.hip"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# Packed float32 instructions are disabled for all device code: the compiler
# may not form them from ordinary float code.
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", INCLUDE, "-I", CSRC]


def _compile(args):
    src, obj, isa_dir = args
    cmd = [hipcc(), *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if isa_dir:
        cmd += ["-save-temps=obj"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(isa_dir: str | None = None, verbose: bool = False) -> str:
    with tempfile.TemporaryDirectory() as tmp:
        work = isa_dir or tmp
        os.makedirs(work, exist_ok=True)
        jobs = [(s, os.path.join(work, s.replace(".hip", ".o")), isa_dir) for s in SOURCES]
        with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
            objs = list(ex.map(_compile, jobs))
        tmp_lib = LIB + ".tmp"
        cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp_lib]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        os.replace(tmp_lib, LIB)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--isa", default=None, help="keep device assembly under this dir")
    a = ap.parse_args(argv)
    print(build(isa_dir=a.isa, verbose=True))


if __name__ == "__main__":
    sys.exit(main())
