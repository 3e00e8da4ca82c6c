"""Randomized GPU parity: seeded random shapes through the whole chain.

Every case draws a legal shape (experts per rank, rank count, k up to 32,
token counts from 1 to a few thousand, bf16 rows of any 16-byte multiple
or fp8 rows with 128-wide scale blocks), a routing (uniform or Zipf-skewed,
with or without unused slots), a work split and sometimes a rank whose
capacity is short, and compares the HIP path with the oracle exactly as the
hand-picked cases do: layout, plan, regions and stand-in expert bit for bit,
y within the combine tolerance.  The same for the per-peer deduplicated
path.  The seeds are fixed, so a failure names its case.
"""
import os

import numpy as np
import pytest

import workloads as wl

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# MOE_RANDOM_CASES=n widens a run to n per-slot and n/2 deduplicated cases.
N_SLOT_CASES = int(os.environ.get("MOE_RANDOM_CASES", "96"))
N_DEDUP_CASES = N_SLOT_CASES // 2
BUDGET = 40_000_000   # T * k * H per case (row bytes the oracle and checks touch)


def _shape(seed, dedup=False):
    rng = np.random.default_rng(1000 + seed)
    R = int(rng.choice([1, 2, 4, 8, 16, 32, 64]))
    L = int(rng.choice([1, 2, 3, 4, 8]))
    while R * L > 1024:
        L = max(1, L // 2)
    E = R * L
    k = int(rng.integers(1, min(32, E) + 1))
    fp8 = bool(rng.random() < 0.3)
    H = 128 * int(rng.integers(1, 65)) if fp8 else 8 * int(rng.integers(1, 1153))
    T = int(np.exp(rng.uniform(0.0, np.log(5000.0))))
    T = max(1, min(T, BUDGET // (k * H)))
    mask = float(rng.choice([0.0, 0.0, 0.1, 0.5]))
    zipf = float(rng.choice([0.0, 1.2]))
    policy = int(rng.choice([0, 3, 4])) if not dedup else 0
    cpolicy = int(rng.choice([0, 3])) if not dedup else 0
    short = bool(rng.random() < 0.25) and not dedup
    return dict(T=T, H=H, E=E, R=R, k=k, payload=wl.FP8_E4M3 if fp8 else wl.BF16, mask=mask,
                zipf=zipf, policy=policy, cpolicy=cpolicy, short=short, seed=seed)


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_26444_amd import moe
    moe.lib()


@pytest.mark.parametrize("seed", range(N_SLOT_CASES))
def test_random_shape_matches_oracle(seed):
    from test_gpu_parity import _full_parity
    s = _shape(seed)
    cfg = wl.custom(s["T"], s["H"], s["E"], s["R"], s["k"], payload=s["payload"],
                    zipf_s=s["zipf"], seed=5000 + seed)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], s["mask"], seed=seed) if s["mask"] else None
    delta = None
    if s["short"]:
        delta = [0] * s["R"]
        delta[seed % s["R"]] = -(1 + seed % 7)
    _full_parity(cfg, inp, idx=idx, policy=s["policy"], combine_policy=s["cpolicy"],
                 cap_delta=delta, spare_rows=1)


@pytest.mark.parametrize("seed", range(N_DEDUP_CASES))
def test_random_shape_dedup_matches_oracle(seed):
    from test_gpu_dedup import _dedup_parity
    s = _shape(100000 + seed, dedup=True)
    cfg = wl.custom(s["T"], s["H"], s["E"], s["R"], s["k"], payload=s["payload"],
                    zipf_s=s["zipf"], seed=6000 + seed)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], s["mask"], seed=seed) if s["mask"] else None
    _dedup_parity(cfg, inp, idx=idx)


N_LARGE_CASES = 4


def _large_shape(seed):
    """A random batch large enough that the default split hands every part
    out at run time (a plan part carries at least 128 KiB on average)."""
    rng = np.random.default_rng(3000 + seed)
    R = int(rng.choice([16, 32, 64]))
    E = R * int(rng.choice([2, 4]))
    k = 8 if seed % 2 == 0 else 6
    fp8 = seed == 2   # fp8 rows: combine claims every part, dispatch's parts are smaller
    H = 128 * int(rng.integers(40, 65)) if fp8 else 8 * int(rng.integers(640, 1025))
    row_b = H if fp8 else 2 * H
    T = int(rng.integers(12000, 20001))
    while T * 2 * H * (1 + k) // 12288 < (128 << 10):   # combine's part bytes
        T += 2048
    return dict(T=T, H=H, E=E, R=R, k=k, fp8=fp8, row_b=row_b,
                mask=float(rng.choice([0.0, 0.05])), zipf=float(rng.choice([0.0, 1.2])))


@pytest.mark.parametrize("seed", range(N_LARGE_CASES))
def test_random_large_batch_matches_oracle(seed):
    from test_gpu_parity import _full_parity
    s = _large_shape(seed)
    cfg = wl.custom(s["T"], s["H"], s["E"], s["R"], s["k"],
                    payload=wl.FP8_E4M3 if s["fp8"] else wl.BF16, zipf_s=s["zipf"],
                    seed=7000 + seed)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], s["mask"], seed=seed) if s["mask"] else None
    _full_parity(cfg, inp, idx=idx, repeat=2, spare_rows=1)
