"""Seeded synthetic inputs for the MoE dispatch/combine path.

This module is the only code shared by the CPU oracle's tests and the GPU
path's tests and benchmark.  It draws inputs and nothing else: it holds none
of the arithmetic of layout, dispatch or combine.  Routing (top-k of logits
and a softmax over the chosen logits) is the router that sits in front of the
operator; it is generated here once, as data, and both sides consume the same
arrays.

Workloads follow the paper's MoE microbenchmark shape (Section 8.1 and
Table 2: 4096 tokens per batch, hidden 7168, top-8 routing) and widen it to prefill-sized,
skewed, fp8 and mid-width cases.  Each workload is a dict of plain integers and
strings; `make_routing` and `make_inputs` turn one into numpy arrays.

Conventions (readings where the paper is silent):
  * one numpy Generator(PCG64(seed)) per workload; logits [T,E] float32 are
    drawn first, then the hidden states [T,H] float32;
  * top-k columns are in descending logit order, ties to the lower expert
    (stable sort); weights are a max-subtracted float32 softmax over the k
    chosen logits;
  * Zipf skew: expert e gets the bias -s*ln(e+1) (rank e+1, no permutation);
  * forced tokens: every token t with t % round(1/frac) == 0 gets
    logit[t, E-1] := max_e logit[t, e] + 1 before top-k;
  * bf16 values are the round-to-nearest-even of the float32 draws;
  * fp8 payloads are OCP E4M3FN with one float32 scale per 128 consecutive
    elements of a row: scale = amax/448 (1 when amax == 0), q = x/scale
    clamped to +-448 and rounded by torch's float8_e4m3fn cast.
"""
from __future__ import annotations

import numpy as np

# Payload dtype codes; they match the library's dtype argument.
BF16 = 0
FP8_E4M3 = 1

FP8_BLOCK = 128

WORKLOADS = {
    # 128 tokens, H=256 bf16, 16 experts over 4 ranks, top-2, identity expert.
    "tiny_t128_h256_e16_r4_k2": dict(
        T=128, H=256, E=16, R=4, k=2, payload=BF16, zipf_s=0.0,
        force_frac=0.0, expert="identity", seed=0),
    # Decode-sized expert-parallel share: 4096 tokens, H=7168, 256 experts
    # over 64 ranks, top-8 of N(0,1) logits.
    "decode_t4096_h7168_e256_r64_k8": dict(
        T=4096, H=7168, E=256, R=64, k=8, payload=BF16, zipf_s=0.0,
        force_frac=0.0, expert="scale", seed=0),
    # Prefill-sized share with Zipf(1.2)-biased routing (hot experts).
    "prefill_zipf1.2_t16384_h7168_e256_r64_k8": dict(
        T=16384, H=7168, E=256, R=64, k=8, payload=BF16, zipf_s=1.2,
        force_frac=0.0, expert="scale", seed=0),
    # fp8 E4M3 payload with per-128 float32 block scales, uniform routing.
    "fp8_t16384_h7168_e256_r64_k8": dict(
        T=16384, H=7168, E=256, R=64, k=8, payload=FP8_E4M3, zipf_s=0.0,
        force_frac=0.0, expert="scale", seed=0),
    # Large mid-width: Zipf(1.5) plus 5% of tokens forced onto one expert.
    "large_zipf1.5_forced_t32768_h4096_e128_r32_k8": dict(
        T=32768, H=4096, E=128, R=32, k=8, payload=BF16, zipf_s=1.5,
        force_frac=0.05, expert="scale", seed=0),
}

# Short aliases used on command lines.
ALIASES = {
    "tiny": "tiny_t128_h256_e16_r4_k2",
    "decode": "decode_t4096_h7168_e256_r64_k8",
    "prefill": "prefill_zipf1.2_t16384_h7168_e256_r64_k8",
    "fp8": "fp8_t16384_h7168_e256_r64_k8",
    "large": "large_zipf1.5_forced_t32768_h4096_e128_r32_k8",
}


def get(name: str) -> dict:
    """Return a copy of a named workload (full name or alias) with its name."""
    full = ALIASES.get(name, name)
    cfg = dict(WORKLOADS[full])
    cfg["name"] = full
    return cfg


def custom(T, H, E, R, k, payload=BF16, zipf_s=0.0, force_frac=0.0,
           expert="scale", seed=0, name=None) -> dict:
    """A workload of arbitrary shape (used for ragged and edge-case tests)."""
    return dict(T=T, H=H, E=E, R=R, k=k, payload=payload, zipf_s=zipf_s,
                force_frac=force_frac, expert=expert, seed=seed,
                name=name or f"custom_t{T}_h{H}_e{E}_r{R}_k{k}_p{payload}")


def row_bytes(cfg) -> int:
    """Bytes of one hidden row as dispatched (bf16: 2H, fp8: H)."""
    return cfg["H"] * (2 if cfg["payload"] == BF16 else 1)


def scale_row_bytes(cfg) -> int:
    """Bytes of one row of fp8 block scales (0 for bf16 payloads)."""
    return 0 if cfg["payload"] == BF16 else (cfg["H"] // FP8_BLOCK) * 4


def _draw_logits(rng, cfg) -> np.ndarray:
    T, E = cfg["T"], cfg["E"]
    logits = rng.standard_normal((T, E), dtype=np.float32)
    if cfg["zipf_s"]:
        bias = (-cfg["zipf_s"] * np.log(np.arange(1, E + 1, dtype=np.float64))
                ).astype(np.float32)
        logits += bias[None, :]
    if cfg["force_frac"]:
        step = int(round(1.0 / cfg["force_frac"]))
        rows = np.arange(0, T, step)
        logits[rows, E - 1] = logits[rows].max(axis=1) + np.float32(1.0)
    return logits


def _route(logits: np.ndarray, k: int):
    T = logits.shape[0]
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    topk_idx = np.ascontiguousarray(order.astype(np.int32))
    chosen = np.take_along_axis(logits, order, axis=1).astype(np.float32)
    m = chosen.max(axis=1, keepdims=True)
    ex = np.exp(chosen - m, dtype=np.float32)
    topk_w = (ex / ex.sum(axis=1, keepdims=True, dtype=np.float32)
              ).astype(np.float32)
    assert topk_idx.shape == (T, k)
    return topk_idx, np.ascontiguousarray(topk_w)


def make_routing(cfg):
    """(topk_idx int32 [T,k], topk_w float32 [T,k]) for a workload."""
    rng = np.random.Generator(np.random.PCG64(cfg["seed"]))
    return _route(_draw_logits(rng, cfg), cfg["k"])


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bf16 bit patterns (inputs finite)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (r >> np.uint32(16)).astype(np.uint16)


def _quantize_fp8(xf: np.ndarray):
    import torch  # CPU only: the float8_e4m3fn cast is the quantizer
    T, H = xf.shape
    blk = xf.reshape(T, H // FP8_BLOCK, FP8_BLOCK)
    amax = np.abs(blk).max(axis=2)
    scale = np.where(amax > 0, amax / np.float32(448.0),
                     np.float32(1.0)).astype(np.float32)
    q = np.clip(blk / scale[:, :, None], -448.0, 448.0).astype(np.float32)
    q8 = torch.from_numpy(q.reshape(T, H)).to(torch.float8_e4m3fn)
    return q8.view(torch.uint8).numpy().copy(), np.ascontiguousarray(scale)


def make_inputs(cfg) -> dict:
    """All inputs of one workload as numpy arrays.

    Keys: topk_idx int32 [T,k]; topk_w float32 [T,k]; x uint16 [T,H] (bf16
    bits) or uint8 [T,H] (fp8 bits); x_scales float32 [T,H/128] or None.
    """
    T, H = cfg["T"], cfg["H"]
    rng = np.random.Generator(np.random.PCG64(cfg["seed"]))
    topk_idx, topk_w = _route(_draw_logits(rng, cfg), cfg["k"])
    xf = rng.standard_normal((T, H), dtype=np.float32)
    if cfg["payload"] == BF16:
        x, xs = f32_to_bf16_bits(xf), None
    else:
        assert H % FP8_BLOCK == 0
        x, xs = _quantize_fp8(xf)
    del xf
    return dict(topk_idx=topk_idx, topk_w=topk_w, x=x, x_scales=xs)


def random_bf16_rows(n_rows: int, H: int, seed: int) -> np.ndarray:
    """Seeded N(0,1) bf16 bit rows [n_rows, H] (stand-in expert outputs)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return f32_to_bf16_bits(rng.standard_normal((n_rows, H), dtype=np.float32))


def mask_slots(topk_idx: np.ndarray, frac: float, seed: int) -> np.ndarray:
    """Copy of topk_idx with a seeded fraction of slots set to -1 (unused)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = topk_idx.copy()
    out[rng.random(out.shape) < frac] = -1
    return out


def region_rows(rank_count) -> list:
    """Rows to reserve per emulated rank region (at least one)."""
    return [max(1, int(c)) for c in rank_count]


def zipf_hot_factor(topk_idx: np.ndarray, E: int) -> float:
    """Load of the hottest expert divided by the mean expert load."""
    cnt = np.bincount(topk_idx[topk_idx >= 0].ravel(), minlength=E)
    return float(cnt.max() / max(1e-9, cnt.mean()))

