"""Host-side logic of bench.py (no GPU): the single-GPU refusal, the
algorithmic byte counts behind `value` and `roofline.achieved`, and the rule
that drops the traffic figure once a kernel's sources change."""
import os

import pytest

import bench
import workloads as wl


def test_more_than_one_gpu_is_refused(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    assert "one GPU" in capsys.readouterr().err


# Bytes per launch computed independently from the per-token definitions:
# dispatch reads x once and writes one row per routed slot plus a 4-byte pos
# per slot; combine reads one bf16 row per slot plus (weight, pos) and writes
# y once.  Expected: those counts at each workload, rounded (bytes).
@pytest.mark.parametrize("name,dispatch,combine,rel", [
    ("tiny", 197.6e3, 198.7e3, 1e-3),
    ("decode", 528.6e6, 528.7e6, 1e-3),
    ("prefill", 2.1145e9, 2.1150e9, 1e-4),
    ("fp8", 1.0905e9, 2.1150e9, 1e-4),
    ("large", 2.417e9, 2.418e9, 1e-3),
])
def test_algorithmic_bytes_per_workload(name, dispatch, combine, rel):
    b = bench.algorithmic_bytes(wl.get(name))
    assert b["dispatch"] == pytest.approx(dispatch, rel=rel)
    assert b["combine"] == pytest.approx(combine, rel=rel)


def test_algorithmic_bytes_per_token_form():
    cfg = wl.custom(T=3, H=256, E=8, R=2, k=2, payload=wl.FP8_E4M3)
    b = bench.algorithmic_bytes(cfg)
    row = 256 + (256 // 128) * 4            # fp8 bytes + block scales
    assert b["row"] == row
    assert b["dispatch"] == 3 * (row * (1 + 2) + 4 * 2)
    assert b["combine"] == 3 * (2 * 256 * (2 + 1) + 8 * 2)


def test_traffic_figure_is_dropped_when_the_kernel_source_changes(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2607_26444_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "dispatch.hip").write_text("kernel v1\n")
    (csrc / "moe_internal.h").write_text("header\n")
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h = bench.kernel_source_hash("dispatch")
    prof = tmp_path / "profiles" / "traffic_dispatch_w.txt"
    prof.write_text(f"# header\nhbm_bytes_per_launch: 1234\nsource_hash: {h}\n")
    assert bench.read_traffic("w", "dispatch") == 1234.0
    (csrc / "dispatch.hip").write_text("kernel v2\n")
    assert bench.read_traffic("w", "dispatch") is None
    (csrc / "dispatch.hip").write_text("kernel v1\n")
    (csrc / "moe_internal.h").write_text("header changed\n")
    assert bench.read_traffic("w", "dispatch") is None
    assert bench.read_traffic("other", "dispatch") is None
