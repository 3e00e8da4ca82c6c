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


def test_read_write_split_adds_up_to_the_kernel_bytes():
    for name in ("tiny", "decode", "prefill", "fp8", "large"):
        b = bench.algorithmic_bytes(wl.get(name))
        assert b["dispatch_read"] + b["dispatch_write"] == b["dispatch"]
        assert b["combine_read"] + b["combine_write"] == b["combine"]
        # every routed slot writes one x row; combine reads k expert rows per
        # written y row (all slots routed in these workloads)
        k = wl.get(name)["k"]
        assert b["dispatch_write"] == k * (b["dispatch_read"] - 4 * b["n"])
        assert b["combine_read"] - 8 * b["n"] == k * b["combine_write"]


def test_stream_ceiling_is_the_time_weighted_rate():
    # equal rates: the ceiling is that rate
    assert bench.stream_ceiling(3e9, 5e9, 6000.0, 6000.0) == pytest.approx(6000.0)
    # 1 GB read at 8000 GB/s (0.125 ms) + 7 GB written at 5000 GB/s (1.4 ms)
    assert bench.stream_ceiling(1e9, 7e9, 8000.0, 5000.0) == pytest.approx(8e9 / 1.525e-3 / 1e9)
    # pure streams give back their own rate
    assert bench.stream_ceiling(0, 2e9, 7000.0, 5000.0) == pytest.approx(5000.0)
    assert bench.stream_ceiling(2e9, 0, 7000.0, 5000.0) == pytest.approx(7000.0)
    # the ceiling lies between the two rates
    c = bench.stream_ceiling(1e9, 1e9, 7000.0, 5000.0)
    assert 5000.0 < c < 7000.0


def test_sampled_steps():
    """Per-phase events: every N-th timed step from the first."""
    assert bench.sampled_steps(100, 4) == list(range(0, 100, 4))
    assert len(bench.sampled_steps(100, bench.EVENT_EVERY)) == 25
    assert bench.sampled_steps(5, 1) == [0, 1, 2, 3, 4]
    assert bench.sampled_steps(5, 0) == [0, 1, 2, 3, 4]
    assert bench.sampled_steps(3, 10) == [0]
