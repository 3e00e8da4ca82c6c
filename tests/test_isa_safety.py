"""Device-code checks on the gfx950 assembly of libmoe (CPU only).

The library's kernels must write memory only through vector instructions:
no scalar-cache stores, scalar atomics or scalar-cache write-back/discard.
They must also use no scratch (private) memory and no flat addressing for
their hot-loop data accesses.
"""
import os
import re
import tempfile

import pytest

from paper_2607_26444_amd import build as libbuild

SCALAR_WRITE = re.compile(
    r"^\s*s_(store|buffer_store|scratch_store|atomic|buffer_atomic|dcache_wb|dcache_discard)")


@pytest.fixture(scope="module")
def isa():
    with tempfile.TemporaryDirectory() as tmp:
        libbuild.build(isa_dir=tmp)
        texts = {}
        for f in os.listdir(tmp):
            if f.endswith(".s") and "gfx950" in f:
                texts[f] = open(os.path.join(tmp, f)).read()
    assert texts
    return texts


def test_no_scalar_memory_writes(isa):
    for name, text in isa.items():
        bad = [ln for ln in text.splitlines() if SCALAR_WRITE.match(ln)]
        assert not bad, (name, bad[:5])


def test_no_scratch(isa):
    for name, text in isa.items():
        sizes = re.findall(r"\.private_segment_fixed_size:\s+(\d+)", text)
        assert all(int(s) == 0 for s in sizes), name


def test_hot_loops_use_global_memory_instructions(isa):
    for name, text in isa.items():
        flat = [ln for ln in text.splitlines() if re.match(r"^\s*flat_(load|store|atomic)", ln)]
        assert not flat, (name, flat[:5])
