"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Layout (counts, offsets, pos, row_src), the partition plan, dispatch (region
bytes, untouched sentinels) and the stand-in expert are compared bit for
bit; combine within |y - y_ref| <= 8e-3*|y_ref| + 1e-3.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import workloads as wl  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_26444_amd import moe
    moe.lib()  # raises if libmoe.so is missing: there is no fallback


def _h():
    import gpu_harness
    return gpu_harness


def _full_parity(cfg, inp=None, idx=None, w=None, spare_rows=2, cap_delta=None,
                 identity=None, scale_pitch=None, policy=0, trace=False, combine_policy=0,
                 repeat=1, capacity=None, waves=0):
    h = _h()
    inp = wl.make_inputs(cfg) if inp is None else inp
    h.log(f"[parity] {cfg['name']} T={cfg['T']} H={cfg['H']} E={cfg['E']} R={cfg['R']} "
          f"k={(idx if idx is not None else inp['topk_idx']).shape[1]}")
    run = h.GpuRun(cfg, inp, topk_idx=idx, topk_w=w, spare_rows=spare_rows,
                   cap_delta=cap_delta, identity=identity, scale_pitch=scale_pitch,
                   policy=policy, trace=trace, combine_policy=combine_policy, repeat=repeat,
                   capacity=capacity, waves=waves)
    ref = h.oracle_chain(cfg, inp, topk_idx=idx, topk_w=w, caps=run.caps,
                         identity=identity, scale_pitch=run.scale_pitch, capacity=capacity)
    # layout: bit-exact
    for key in ("expert_count", "expert_offset", "rank_count", "rank_offset", "pos",
                "row_src"):
        assert np.array_equal(run.layout[key], ref["layout"][key]), key
    T, k = run.idx.shape
    assert np.array_equal(run.plan, oracle.plan(ref["layout"]["pos"], T, k,
                                                len(run.plan) - 1)), "plan"
    # dispatch: bit-exact region bytes, sentinels untouched
    h.check_regions(run, run.regions, ref["regs"])
    if run.sregions is not None:
        h.check_regions(run, run.sregions, ref["sregs"])
    # stand-in expert: bit-exact
    written = np.minimum(ref["layout"]["rank_count"], run.caps) if capacity is None \
        else run.caps   # fixed windows: the stand-in expert runs over whole windows
    h.check_regions(run, run.eregions,
                    [e.view(np.uint8).reshape(e.shape[0], 2 * e.shape[1]) for e in ref["ey"]],
                    written)
    # combine: tolerance
    ok, msg = h.combine_close(run.y, ref["y"])
    assert ok, msg
    assert run.layout["status"] == ref["layout"]["status"] | ref["status"], \
        (run.layout["status"], ref["layout"]["status"], ref["status"])
    h.log(f"[parity] {cfg['name']} ok ({msg})")
    return run, ref


def test_library_is_native_and_single_runtime():
    """libmoe.so is loaded and shares torch's HIP runtime (one copy)."""
    from paper_2607_26444_amd import moe
    moe.lib()
    maps = open("/proc/self/maps").read()
    assert "libmoe.so" in maps
    hip = {line.split()[-1] for line in maps.splitlines() if "libamdhip64" in line}
    assert len(hip) == 1, hip


def test_tiny_workload():
    _full_parity(wl.get("tiny"))


def test_tiny_identity_softmax_returns_x():
    """Identity expert with softmax weights: y == x bit for bit."""
    h = _h()
    cfg = wl.get("tiny")
    inp = wl.make_inputs(cfg)
    run = h.GpuRun(cfg, inp)
    assert np.array_equal(run.y, inp["x"])


@pytest.mark.parametrize("T,H,E,R,k,payload,mask", [
    (1000, 1032, 24, 6, 3, wl.BF16, 0.1),      # ragged chunks, segments and batches
    (777, 7168, 64, 16, 8, wl.BF16, 0.0),
    (700, 640, 32, 8, 5, wl.FP8_E4M3, 0.05),   # 20-byte scale rows
    (513, 4096, 128, 32, 8, wl.FP8_E4M3, 0.0),
    (300, 256, 16, 4, 1, wl.BF16, 0.0),        # k = 1
    (200, 512, 64, 8, 16, wl.BF16, 0.2),       # k = 16
    (150, 264, 64, 4, 32, wl.BF16, 0.3),       # k = 32
    (400, 128, 16, 1, 4, wl.BF16, 0.0),        # R = 1
    (400, 128, 16, 16, 4, wl.BF16, 0.0),       # R = E
    (1, 8, 4, 2, 2, wl.BF16, 0.0),             # one token, one 16-byte segment
    (2049, 2048, 256, 64, 8, wl.BF16, 0.0),
    (256, 512, 32, 8, 4, wl.BF16, 0.1),        # largest single-kernel layout
    (257, 512, 32, 8, 4, wl.BF16, 0.1),        # smallest two-kernel layout
    (300, 2048, 16, 4, 2, wl.FP8_E4M3, 0.0),   # 64-byte scale rows
    (2000, 256, 1024, 64, 8, wl.BF16, 0.05),   # MOE_MAX_EXPERTS
    (300, 16384, 64, 8, 4, wl.BF16, 0.0),      # 32 KiB rows: two 16 KiB passes
    (100, 20480, 32, 8, 2, wl.FP8_E4M3, 0.0),  # 20 KiB fp8 rows, 640-byte scale rows
    (131072, 128, 256, 64, 8, wl.BF16, 0.0),   # 1M slots, 128 layout chunks
    (90, 8192, 64, 16, 6, wl.FP8_E4M3, 0.1),   # 256-byte scale rows, k=6
    (64, 1152, 1024, 256, 8, wl.BF16, 0.0),    # maximum expert count
    (96, 1152, 1024, 1024, 8, wl.BF16, 0.1),   # one expert per rank at the maximum: full rank tables
])
def test_custom_shapes(T, H, E, R, k, payload, mask):
    cfg = wl.custom(T, H, E, R, k, payload=payload, seed=T + H)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], mask, seed=T) if mask else None
    _full_parity(cfg, inp, idx=idx)


@pytest.mark.parametrize("T,H,E,R,k,mask,cap", [
    (300, 4104, 32, 8, 2, 0.1, False),    # 8 KiB + 16 B: one lane in the last segment
    (257, 6152, 64, 16, 4, 0.2, True),    # 12 KiB + 16 B, capacity drops
    (129, 7176, 256, 64, 7, 0.05, False),  # slot width 8 with one pad slot, ragged tail
    (200, 8192, 64, 16, 8, 0.1, True),    # 16 KiB: every register segment used
    (200, 4096, 64, 16, 8, 0.1, False),   # 8 KiB: segment-by-segment path, just below
    (200, 8200, 64, 16, 8, 0.1, False),   # 16 KiB + 16 B: segment-by-segment, just above
])
def test_combine_row_widths(T, H, E, R, k, mask, cap):
    """Combine output rows around the widths that are reduced into registers
    and stored as one burst (more than 8, at most 16 KiB): ragged last
    segments, masked and capacity-dropped slots, both neighbours."""
    cfg = wl.custom(T, H, E, R, k, zipf_s=1.2, seed=T + H + k)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], mask, seed=T) if mask else None
    delta = None
    if cap:
        delta = [0] * R
        delta[0] = -7
    _full_parity(cfg, inp, idx=idx, cap_delta=delta, spare_rows=1)


@pytest.mark.parametrize("pitch", [0, 116, 128, 256])
def test_fp8_scale_pitch(pitch):
    """Scale rows (112 bytes here) packed (pitch 0) or pitched: scales then
    zeros to the pitch; 116 takes the 4-byte path."""
    cfg = wl.custom(333, 3584, 64, 16, 8, payload=wl.FP8_E4M3, seed=77)
    _full_parity(cfg, scale_pitch=pitch)


def test_fp8_scale_pitch_too_small_is_rejected():
    from paper_2607_26444_amd import moe
    h = _h()
    cfg = wl.custom(16, 3584, 64, 16, 8, payload=wl.FP8_E4M3, seed=78)
    with pytest.raises(moe.MoeError) as ei:
        h.GpuRun(cfg, wl.make_inputs(cfg), scale_pitch=64)
    assert ei.value.code == moe.MOE_EINVAL


@pytest.mark.parametrize("policy", [1, 2])
@pytest.mark.parametrize("T,H,E,R,k,payload,mask", [
    (1000, 1032, 24, 6, 3, wl.BF16, 0.1),
    (700, 640, 32, 8, 5, wl.FP8_E4M3, 0.05),
    (2049, 7168, 256, 64, 8, wl.BF16, 0.0),
    (513, 4096, 128, 32, 8, wl.FP8_E4M3, 0.0),
])
def test_pull_policies_match_oracle(policy, T, H, E, R, k, payload, mask):
    """The pull work splits (rows even, or a fixed wavefront group per rank)
    give the same bytes as the oracle, with a capacity overflow on one rank."""
    cfg = wl.custom(T, H, E, R, k, payload=payload, seed=T + 1)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], mask, seed=T) if mask else None
    delta = [0] * R
    delta[1] = -3
    run, _ = _full_parity(cfg, inp, idx=idx, policy=policy, cap_delta=delta, spare_rows=1)


@pytest.mark.parametrize("T,H,E,R,k,payload,mask", [
    (1000, 1032, 24, 6, 3, wl.BF16, 0.1),
    (700, 640, 32, 8, 5, wl.FP8_E4M3, 0.05),
    (3000, 7168, 256, 64, 8, wl.BF16, 0.0),
    (100, 256, 16, 4, 2, wl.BF16, 0.0),
    (300, 1152, 1024, 1024, 8, wl.FP8_E4M3, 0.1),   # claimed parts with 1024 rank-table entries
])
def test_dynamic_policy_matches_oracle(T, H, E, R, k, payload, mask):
    """Parts handed out at run time: same bytes for dispatch, same y for
    combine; three calls on one layout exercise the ticket reset."""
    cfg = wl.custom(T, H, E, R, k, payload=payload, zipf_s=1.2, seed=T + 2)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], mask, seed=T) if mask else None
    _full_parity(cfg, inp, idx=idx, policy=3, combine_policy=3, repeat=3)
    # the default split hands out its second half at run time: same reset
    _full_parity(cfg, inp, idx=idx, policy=0, combine_policy=0, repeat=3)


@pytest.mark.parametrize("policy,cpolicy", [(0, 0), (1, 0), (2, 0), (3, 3), (4, 4)])
@pytest.mark.parametrize("waves", [64, 256, 3072])
def test_explicit_wave_counts_match_oracle(policy, cpolicy, waves):
    """Every work split gives the oracle's bytes and y at a chosen wavefront
    count, below and above what the device holds at once (64 wavefronts use
    two of the four ticket shards)."""
    T, H, E, R, k = 2500, 1536, 64, 16, 6
    cfg = wl.custom(T, H, E, R, k, zipf_s=1.2, seed=waves + policy)
    _full_parity(cfg, policy=policy, combine_policy=cpolicy, waves=waves, repeat=2)


@pytest.mark.parametrize("waves", [4, 96])
def test_claims_with_fewer_wavefronts_than_shards(waves):
    """Claiming every part with 4 or 96 wavefronts, which fill one or three
    runs of 32 and so use one or three ticket shards: every shard in use has
    wavefronts, so no claim is left untaken."""
    T, H, E, R, k = 1500, 2048, 64, 16, 8
    cfg = wl.custom(T, H, E, R, k, zipf_s=1.2, seed=waves)
    _full_parity(cfg, policy=3, combine_policy=3, waves=waves, repeat=2)


@pytest.mark.parametrize("cpolicy,waves", [(0, 64), (0, 3072), (3, 256), (3, 3072)])
def test_combine_burst_rows_at_explicit_wave_counts(cpolicy, waves):
    """12 KiB output rows (stored from registers) under both combine splits,
    with fewer wavefronts than CUs and more than fit on the device at once."""
    cfg = wl.custom(1500, 6144, 64, 16, 8, zipf_s=1.2, seed=waves + cpolicy)
    inp = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp["topk_idx"], 0.05, seed=waves)
    _full_parity(cfg, inp, idx=idx, combine_policy=cpolicy, waves=waves, repeat=2)


@pytest.mark.parametrize("T,H,E,R,k,payload,C,zipf", [
    (1000, 1032, 24, 6, 3, wl.BF16, 200, 0.0),      # ample windows
    (1000, 1032, 24, 6, 3, wl.BF16, 60, 1.2),       # hot experts overflow
    (700, 640, 32, 8, 5, wl.FP8_E4M3, 90, 1.2),
    (4096, 7168, 256, 64, 8, wl.BF16, 160, 0.0),    # decode-sized share
    (200, 256, 16, 4, 2, wl.BF16, 0, 0.0),          # zero capacity: nothing placed
    (100, 512, 16, 4, 4, wl.BF16, 7, 0.0),          # single-kernel layout
])
def test_fixed_capacity_layout(T, H, E, R, k, payload, C, zipf):
    cfg = wl.custom(T, H, E, R, k, payload=payload, zipf_s=zipf, seed=T + C)
    inp = wl.make_inputs(cfg)
    run, ref = _full_parity(cfg, inp, capacity=C)
    overflow = (ref["layout"]["status"] & 4) != 0
    assert overflow == bool((np.bincount(inp["topk_idx"].ravel(), minlength=E) > C).any())


def test_fixed_capacity_step_in_a_captured_graph():
    """layout_fixed -> dispatch -> combine captured once and replayed; each
    replay (with eager work in between) matches the eager result."""
    from paper_2607_26444_amd import moe
    cfg = wl.custom(2048, 7168, 256, 64, 8, zipf_s=1.2, seed=9)
    inp = wl.make_inputs(cfg)
    T, H, E, R, k, C = 2048, 7168, 256, 64, 8, 256
    L = E // R
    dev = "cuda"
    x_d = torch.from_numpy(np.ascontiguousarray(inp["x"]).view(np.int16)).to(dev)
    idx_d = torch.from_numpy(inp["topk_idx"]).to(dev)
    w_d = torch.from_numpy(inp["topk_w"]).to(dev)
    lay = moe.Layout(T, k, E, R, capacity=C)
    regions = moe.Regions([L * C] * R, 2 * H)
    y = torch.zeros((T, H), dtype=torch.int16, device=dev)

    def step():
        lay.run(idx_d)
        moe.moe_dispatch(x_d, None, 0, H, E, R, idx_d, lay.pos, lay.rank_offset,
                         regions.table, None, regions.cap, lay.workspace, lay.status)
        moe.moe_combine(regions.table, w_d, H, E, R, idx_d, lay.pos, lay.rank_offset,
                        regions.cap, y, lay.workspace, lay.status)

    step()
    torch.cuda.synchronize()
    eager = y.clone()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()          # warm the occupancy cache on this stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    for i in range(4):
        y.fill_(0)
        lay.pos.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, eager), i
    # Zipf(1.2) sends ~2000 of the 16384 slots to the hottest expert, far
    # above the 256-row windows: those slots are dropped and flagged
    assert int(lay.status.item()) == moe.MOE_STATUS_CAPACITY


def test_trace_records_every_wavefront():
    from paper_2607_26444_amd import moe
    h = _h()
    cfg = wl.custom(3000, 7168, 256, 64, 8, zipf_s=1.2, seed=5)
    run = h.GpuRun(cfg, wl.make_inputs(cfg), trace=True)
    for tr in (run.dtrace, run.ctrace):
        t = tr.view(-1, 2).cpu().numpy()
        used = t[:, 0] != 0
        n = int(used.sum())                # one record per launched wavefront:
        assert np.all(used[:n])            # wavefronts 0 .. W-1, W a power of two
        assert n >= 256 and n & (n - 1) == 0 and moe.MOE_PLAN_PARTS % n == 0
        assert np.all(t[used, 1] >= t[used, 0])
        assert np.all(t[~used] == 0)
        span = t[used, 1].max() - t[used, 0].min()
        assert 0 < span < 10 ** 9


def test_all_slots_unused():
    cfg = wl.custom(100, 64, 8, 2, 2, seed=1)
    inp = wl.make_inputs(cfg)
    idx = -np.ones_like(inp["topk_idx"])
    run, _ = _full_parity(cfg, inp, idx=idx)
    assert np.all(run.y == 0)


def test_capacity_overflow_sets_status_and_drops_rows():
    cfg = wl.custom(600, 256, 16, 4, 4, seed=2)
    inp = wl.make_inputs(cfg)
    run, ref = _full_parity(cfg, inp, spare_rows=0, cap_delta=[-5, 0, -100000, 3])
    assert run.layout["status"] & 4


def test_bad_and_duplicate_indices():
    cfg = wl.custom(300, 128, 16, 4, 4, seed=3)
    inp = wl.make_inputs(cfg)
    idx = inp["topk_idx"].copy()
    idx[3, 1] = 16          # out of range
    idx[7, 2] = -5          # out of range
    idx[11, 3] = idx[11, 0]  # repeat within a row
    run, _ = _full_parity(cfg, inp, idx=idx)
    assert run.layout["status"] == 3


def test_zero_tokens():
    from paper_2607_26444_amd import moe
    lay = moe.Layout(0, 8, 256, 64)
    idx = torch.empty((0, 8), dtype=torch.int32, device="cuda")
    lay.run(idx)
    torch.cuda.synchronize()
    assert lay.expert_count.sum().item() == 0
    assert lay.expert_offset.abs().sum().item() == 0
    assert lay.rank_offset.abs().sum().item() == 0
    assert lay.plan().abs().sum().item() == 0


def test_layout_deterministic():
    from paper_2607_26444_amd import moe
    cfg = wl.get("prefill")
    idx, _ = wl.make_routing(cfg)
    idx_d = torch.from_numpy(idx).cuda()
    outs = []
    for _ in range(3):
        lay = moe.Layout(cfg["T"], cfg["k"], cfg["E"], cfg["R"])
        lay.run(idx_d)
        torch.cuda.synchronize()
        outs.append((lay.pos.cpu().numpy(), lay.row_src.cpu().numpy(), lay.plan().cpu().numpy()))
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(a, b)


def test_decode_workload_full():
    _full_parity(wl.get("decode"))


@pytest.mark.parametrize("name", ["prefill", "fp8", "large"])
def test_full_size_workloads(name):
    """Full-size workloads against the whole oracle chain: layout, plan,
    dispatch and the stand-in expert bit-exact, and combine within the
    tolerance on every token.  Dispatch and combine run twice on one layout
    (at these sizes the default split claims parts at run time, so the
    second call relies on the first one's counter reset; the outputs are
    reset to the sentinel in between).  For bf16 payloads, unit weights on
    the dispatched rows themselves must also give exactly bf16(k*x) for
    every token."""
    h = _h()
    cfg = wl.get(name)
    inp = wl.make_inputs(cfg)
    k = cfg["k"]
    h.log(f"[full] {cfg['name']}")
    run, ref = _full_parity(cfg, inp, spare_rows=1, repeat=2)
    assert run.layout["status"] == 0
    h.log(f"[full] {cfg['name']}: layout, plan, dispatch, expert bit-exact; "
          f"combine within tolerance on all {cfg['T']} tokens")
    del ref

    if cfg["payload"] != wl.FP8_E4M3:
        run1 = h.GpuRun(cfg, inp, topk_w=np.ones_like(inp["topk_w"]),
                        combine_on_dispatch=True)
        xf = (inp["x"].astype(np.uint32) << 16).view(np.float32) * np.float32(k)
        want = h.f32_bits_to_bf16_rne(xf)
        # the sum starts from +0, so a token whose x is -0 gets +0
        want[want == 0x8000] = 0
        bad = run1.y != want
        assert not bad.any(), (int(bad.sum()), run1.y[bad][:8], want[bad][:8])
        h.log(f"[full] {cfg['name']} unit-weight combine == bf16(k*x) exactly")
