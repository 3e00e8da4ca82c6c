"""Golden fixtures: a hand-worked placement example and the paper's Table 2."""
import json
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_layout_worked_example():
    g = _load("layout_worked_example.json")
    idx = np.array(g["topk_idx"], np.int32)
    lay = oracle.layout(idx, g["E"], g["R"])
    for key in ("expert_count", "expert_offset", "rank_count", "rank_offset",
                "pos", "row_src"):
        assert lay[key].tolist() == g[key], key
    assert lay["status"] == 0
    bound = oracle.plan(lay["pos"], g["T"], g["k"], g["plan_P"])
    assert bound.tolist() == g["plan_bound"]
    # dispatch of one-byte rows holding the token id shows the region contents
    x = np.arange(g["T"], dtype=np.uint8).reshape(-1, 1)
    regs, _, st = oracle.dispatch(x, None, idx, lay["pos"], lay["rank_offset"],
                                  g["E"], g["R"], lay["rank_count"])
    assert st == 0
    assert [r.ravel().tolist() for r in regs] == g["region_tokens"]


def test_table2_reading():
    """Our reading of Table 2 reproduces the ratios the text states (this
    checks the reading of the metric's context, not the code)."""
    g = _load("table2_bus_bandwidth.json")
    rows, c = g["rows"], g["claims"]
    gains = [100 * (v[3] / v[2] - 1) for v in rows.values()]
    assert round(min(gains), 1) == c["stratacl_over_zerocopy_min_pct"]
    assert round(max(gains), 1) == c["stratacl_over_zerocopy_max_pct"]
    ht = [100 * (rows[r][2] / rows[r][1] - 1) for r in ("dispatch_ht", "combine_ht")]
    ll = [100 * (rows[r][2] / rows[r][1] - 1) for r in ("dispatch_ll", "combine_ll")]
    assert abs(np.mean(ht) - c["zerocopy_gain_ht_avg_pct"]) < 0.1
    assert abs(np.mean(ll) - c["zerocopy_gain_ll_avg_pct"]) < 0.1
    assert round(np.mean([v[1] / v[0] for v in rows.values()]), 1) == c["cann_over_deepep_avg"]
