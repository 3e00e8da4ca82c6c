"""Every plausible mistake planted in the oracle fails at least one pin.

Each mutant is a copy of oracle/moe_oracle.cpp with one textual change (a
dropped term, an off-by-one, a wrong index or sign, a wrong rounding), built
with g++ into a temporary directory and run against all pins in a child
process.  The real oracle is never modified.
"""
import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "moe_oracle.cpp")

# (name, original fragment, planted mistake)
MUTANTS = [
    ("bf16_round_truncates", "std::nearbyint(std::ldexp(ax, -q))",
     "std::trunc(std::ldexp(ax, -q))"),
    ("bf16_round_ties_away", "std::nearbyint(std::ldexp(ax, -q))",
     "std::round(std::ldexp(ax, -q))"),
    ("bf16_one_bit_too_many", "int q = (e < -126 ? -126 : e) - 7;",
     "int q = (e < -126 ? -126 : e) - 8;"),
    ("bf16_no_subnormal_floor", "int q = (e < -126 ? -126 : e) - 7;",
     "int q = e - 7;"),
    ("fp8_bias_off_by_one", "std::ldexp(1.0 + m / 8.0, ex - 7)",
     "std::ldexp(1.0 + m / 8.0, ex - 8)"),
    ("fp8_subnormal_scale", "std::ldexp((double)m, -9)", "std::ldexp((double)m, -10)"),
    ("layout_misses_duplicates", "for (int32_t jj = 0; jj < j; ++jj)",
     "for (int32_t jj = 0; jj + 1 < j; ++jj)"),
    ("layout_accepts_index_E", "if (e < -1 || e >= E)", "if (e < -1 || e > E)"),
    ("layout_rank_offset_wrong_expert", "rank_offset[r] = expert_offset[r * L];",
     "rank_offset[r] = expert_offset[r];"),
    ("layout_rank_count_drops_expert", "e < (r + 1) * L; ++e) rank_count",
     "e + 1 < (r + 1) * L; ++e) rank_count"),
    ("layout_slot_major_order", "for (int64_t t = 0; t < T; ++t) {\n    for (int32_t j = 0; j < k; ++j) {\n      int64_t s = t * k + j;",
     "for (int32_t j = 0; j < k; ++j) {\n    for (int64_t t = 0; t < T; ++t) {\n      int64_t s = t * k + j;"),
    ("layout_row_src_stores_token", "row_src[p] = (int32_t)s;", "row_src[p] = (int32_t)(s / k);"),
    ("layout_token_order_reversed", "for (int64_t t = 0; t < T; ++t) {\n    for (int32_t j = 0; j < k; ++j) {\n      int64_t s = t * k + j;",
     "for (int64_t t = T - 1; t >= 0; --t) {\n    for (int32_t j = 0; j < k; ++j) {\n      int64_t s = t * k + j;"),
    ("fixed_keeps_overflow", "if (expert_count[e] >= C) { st |= kCapacity; continue; }",
     "if (expert_count[e] >= C + 1) { st |= kCapacity; continue; }"),
    ("fixed_window_reversed", "const int32_t p = e * C + expert_count[e];",
     "const int32_t p = e * C + (C - 1 - expert_count[e]);"),
    ("plan_cost_ignores_read", "int64_t c = 1;", "int64_t c = 0;"),
    ("plan_counts_unused_slots", "c += pos[t * k + j] >= 0 ? 1 : 0;", "c += 1;"),
    ("plan_boundary_off_by_one", "a[(size_t)t] * P < p * A", "a[(size_t)t] * P <= p * A"),
    ("dispatch_short_copy", "x + t * row_bytes, (size_t)row_bytes);",
     "x + t * row_bytes, (size_t)row_bytes - 2);"),
    ("dispatch_scales_from_token0", "x_scales + t * scale_row_bytes, (size_t)scale_row_bytes",
     "x_scales + 0 * t * scale_row_bytes, (size_t)scale_row_bytes"),
    ("expert_scale_off_by_one", "1.0f + 0.01f * (float)e", "1.0f + 0.01f * (float)(e + 1)"),
    ("expert_fp8_block_zero", "local * scale_pitch + (h / 128) * 4", "local * scale_pitch + 0 * h"),
    ("dispatch_scale_pad_not_zeroed", "for (int64_t b = scale_row_bytes; b < scale_pitch; ++b) srow[b] = 0;",
     "for (int64_t b = scale_row_bytes; b < scale_pitch; ++b) srow[b] = srow[b];"),
    ("expert_fp8_scale_dropped", "float dq = oracle_fp8e4m3_to_float(in[h]) * sc;",
     "float dq = oracle_fp8e4m3_to_float(in[h]) * (sc > 0 ? 1.0f : 1.0f);"),
    ("combine_drops_weight", "acc[(size_t)h] += w * oracle_bf16_to_double(row[h]);",
     "acc[(size_t)h] += oracle_bf16_to_double(row[h]);"),
    ("combine_weight_of_slot0", "double w = (double)topk_w[t * k + j];",
     "double w = (double)topk_w[t * k];"),
    ("combine_subtracts", "acc[(size_t)h] += w * oracle_bf16_to_double(row[h]);",
     "acc[(size_t)h] -= w * oracle_bf16_to_double(row[h]);"),
    ("combine_last_slot_dropped", "for (int32_t j = 0; j < k; ++j) {\n      int32_t p = pos[t * k + j];\n      if (p < 0) continue;\n      int32_t r = topk_idx[t * k + j] / L;\n      int64_t local = (int64_t)p - rank_offset[r];\n      if (local >= recv_cap[r]) { st |= kCapacity; continue; }\n      const uint16_t*",
     "for (int32_t j = 0; j + 1 < k; ++j) {\n      int32_t p = pos[t * k + j];\n      if (p < 0) continue;\n      int32_t r = topk_idx[t * k + j] / L;\n      int64_t local = (int64_t)p - rank_offset[r];\n      if (local >= recv_cap[r]) { st |= kCapacity; continue; }\n      const uint16_t*"),
    ("dedup_pairs_by_expert", "if (used[(size_t)jj] && topk_idx[t * k + jj] / L == e / L) seen = true;",
     "if (used[(size_t)jj] && topk_idx[t * k + jj] == e) seen = true;"),
    ("dedup_counts_unused_slots", "if (used[(size_t)jj] && topk_idx[t * k + jj] / L == e / L) seen = true;",
     "if (topk_idx[t * k + jj] / L == e / L) seen = true;"),
    ("dedup_rows_reverse_token_order", "for (int64_t s = 0; s < S; ++s) {     // s = t*k + j ascending",
     "for (int64_t s = S - 1; s >= 0; --s) {     // s = t*k + j ascending"),
    ("dedup_offset_inclusive", "tok_offset[r + 1] = tok_offset[r] + tok_count[r];",
     "tok_offset[r + 1] = tok_offset[r] + tok_count[r] + (r == 0);"),
    ("expand_any_peer_row", "if (tok_pos[s] >= 0 && topk_idx[s] / L == r) return tok_pos[s];",
     "if (tok_pos[s] >= 0) return tok_pos[s];"),
    ("expand_scale_pad_kept", "std::memset(srow + scale_row_bytes, 0, (size_t)(scale_pitch - scale_row_bytes));",
     ";"),
    ("combine_local_all_peers", "if (p < 0 || topk_idx[t * k + j] / L != r) continue;",
     "if (p < 0) continue;"),
    ("combine_local_skips_first", "for (int32_t j = j0; j < k; ++j) {", "for (int32_t j = j0 + 1; j < k; ++j) {"),
    ("combine_local_unweighted", "const double w = (double)topk_w[t * k + j];",
     "const double w = 1.0;"),
    ("combine_no_capacity_flag", "if (local >= recv_cap[r]) { st |= kCapacity; continue; }\n      const uint16_t*",
     "if (local >= recv_cap[r]) { continue; }\n      const uint16_t*"),
]

RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle
oracle.use_library({lib!r})
import oracle_pins as pins
for pin in pins.ALL_PINS:
    try:
        pin()
    except Exception as exc:
        print("CAUGHT_BY", pin.__name__, type(exc).__name__)
        sys.exit(0)
print("NOT_CAUGHT")
"""


def _run_mutant(args):
    name, before, after, tmp = args
    src = open(SRC).read()
    assert src.count(before) >= 1, f"{name}: fragment not found"
    mutated = src.replace(before, after, 1)
    assert mutated != src
    cpp = os.path.join(tmp, f"{name}.cpp")
    lib = os.path.join(tmp, f"lib{name}.so")
    with open(cpp, "w") as f:
        f.write(mutated)
    subprocess.run(["g++", "-O1", "-std=c++17", "-ffp-contract=off", "-shared",
                    "-fPIC", cpp, "-o", lib], check=True)
    code = RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"), lib=lib)
    env = dict(os.environ, OMP_NUM_THREADS="1")
    out = subprocess.run([sys.executable, "-c", code], capture_output=True,
                         text=True, timeout=300, env=env)
    return name, out.returncode, out.stdout + out.stderr[-2000:]


def test_every_mutant_fails_a_pin():
    with tempfile.TemporaryDirectory() as tmp:
        jobs = [(n, b, a, tmp) for (n, b, a) in MUTANTS]
        with cf.ThreadPoolExecutor(max_workers=4) as ex:
            results = list(ex.map(_run_mutant, jobs))
    survivors = [(n, rc, out[-500:]) for (n, rc, out) in results
                 if "CAUGHT_BY" not in out]
    assert not survivors, survivors


@pytest.mark.parametrize("name,before,after", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_fragment_present(name, before, after):
    """Keeps the mutant list in step with the oracle source."""
    assert open(SRC).read().count(before) >= 1
