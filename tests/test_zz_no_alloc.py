"""moe_layout_scratch, the layout that uses the library's own workspace
(for callers that cannot allocate), against moe_layout with a caller
workspace: bit-identical layout outputs and plan, and dispatch + combine
driven by either workspace give identical regions and y, matching the
oracle.  Two calls in a row, the second on a smaller batch, so the second
one runs over what the first left in the library's array.
"""
import ctypes

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
    moe.lib()


def _hip_runtime():
    """The HIP runtime already loaded in this process (torch's), by path."""
    paths = {ln.split()[-1] for ln in open("/proc/self/maps") if "libamdhip64" in ln}
    assert len(paths) == 1, paths
    return ctypes.CDLL(paths.pop())


def _read_device(ptr, nbytes):
    hip = _hip_runtime()
    hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    hip.hipMemcpy.restype = ctypes.c_int
    out = np.empty(nbytes, np.uint8)
    torch.cuda.synchronize()
    assert hip.hipMemcpy(out.ctypes.data, ptr, nbytes, 2) == 0   # device to host
    return out


def _step(h, moe, cfg, inp, idx_d, w_d, x_d, lay_out, ws, caps):
    """dispatch -> stand-in expert -> combine of one batch with the given
    layout outputs and workspace; returns (regions, y)."""
    T, H, E, R, k = cfg["T"], cfg["H"], cfg["E"], cfg["R"], cfg["k"]
    rows = [int(c) for c in caps]
    regions = moe.Regions(rows, wl.row_bytes(cfg), guard_bytes=h.GUARD, fill=h.SENTINEL)
    eregions = moe.Regions(rows, 2 * H, guard_bytes=h.GUARD, fill=h.SENTINEL)
    cap_d = h.to_dev(caps)
    y = torch.full((T, H), 0x5A5A, dtype=torch.int16, device="cuda")
    moe.moe_dispatch(x_d, None, moe.MOE_DTYPE_BF16, H, E, R, idx_d, lay_out["pos"],
                     lay_out["rank_offset"], regions.table, None, cap_d, ws,
                     lay_out["status"])
    moe.moe_expert_scale(regions.table, None, moe.MOE_DTYPE_BF16, H, E, R, False,
                         lay_out["expert_offset"], lay_out["rank_offset"], cap_d,
                         eregions.table, T * k)
    moe.moe_combine(eregions.table, w_d, H, E, R, idx_d, lay_out["pos"],
                    lay_out["rank_offset"], cap_d, y, ws, lay_out["status"])
    torch.cuda.synchronize()
    return regions, y.cpu().numpy().view(np.uint16)


KEYS = ("expert_count", "expert_offset", "rank_count", "rank_offset", "pos", "row_src")


def test_layout_scratch_matches_layout_twice():
    import gpu_harness as h
    from paper_2607_26444_amd import moe
    shapes = [
        # parts of >= 128 KiB: dispatch and combine claim every part
        dict(T=12288, H=7168, E=256, R=64, k=8, zipf=1.2, mask=0.0),
        # smaller batch: the single-workgroup layout, masked slots
        dict(T=200, H=1032, E=32, R=8, k=4, zipf=0.0, mask=0.1),
    ]
    for call, s in enumerate(shapes):
        T, H, E, R, k = s["T"], s["H"], s["E"], s["R"], s["k"]
        cfg = wl.custom(T, H, E, R, k, zipf_s=s["zipf"], seed=40 + call,
                        name=f"no_alloc_{call}")
        inp = wl.make_inputs(cfg)
        idx = wl.mask_slots(inp["topk_idx"], s["mask"], seed=T) if s["mask"] else \
            inp["topk_idx"]
        inp = dict(inp, topk_idx=idx)
        h.log(f"[no-alloc] call {call}: T={T} H={H} E={E} R={R} k={k}")
        idx_d = h.to_dev(idx.astype(np.int32))
        w_d = h.to_dev(inp["topk_w"].astype(np.float32))
        x_d = h.to_dev(h.u8_rows(inp["x"]))

        # the existing entry point with a caller workspace
        lay = moe.Layout(T, k, E, R)
        lay.run(idx_d)
        # the no-allocation variant, outputs in separate buffers
        i32 = dict(dtype=torch.int32, device="cuda")
        out = dict(expert_count=torch.full((E,), -9, **i32),
                   expert_offset=torch.full((E + 1,), -9, **i32),
                   rank_count=torch.full((R,), -9, **i32),
                   rank_offset=torch.full((R + 1,), -9, **i32),
                   pos=torch.full((T * k,), -9, **i32),
                   row_src=torch.full((T * k,), -9, **i32),
                   status=torch.zeros(1, **i32))
        ws = moe.moe_layout_scratch(idx_d, E, R, out["expert_count"], out["expert_offset"],
                                    out["rank_count"], out["rank_offset"], out["pos"],
                                    out["row_src"], out["status"])
        torch.cuda.synchronize()
        assert ws.nbytes == moe.moe_layout_workspace_bytes(T, k, E, R)
        assert ws.ptr % 256 == 0
        for key in KEYS:
            assert torch.equal(out[key], getattr(lay, key)[: out[key].numel()]), key
        assert int(out["status"].item()) == int(lay.status.item())
        plan = _read_device(ws.ptr, (moe.MOE_PLAN_PARTS + 1) * 4).view(np.int32)
        assert np.array_equal(plan, lay.plan().cpu().numpy()), "plan"
        ref_lay = oracle.layout(idx, E, R)
        for key in KEYS:
            assert np.array_equal(out[key].cpu().numpy(), ref_lay[key]), key

        # dispatch -> expert -> combine driven by each workspace
        caps = lay.rank_count.cpu().numpy().astype(np.int32) + 1
        lay_out = dict(out)
        regions_s, y_s = _step(h, moe, cfg, inp, idx_d, w_d, x_d, lay_out, ws, caps)
        tick = h.ticket_words(_read_device(ws.ptr + h.TICKET_OFFSET, h.TICKET_BYTES).view(np.int32))
        assert not tick.any(), tick
        lay_ref = dict(pos=lay.pos, rank_offset=lay.rank_offset,
                       expert_offset=lay.expert_offset, status=lay.status)
        regions_w, y_w = _step(h, moe, cfg, inp, idx_d, w_d, x_d, lay_ref, lay.workspace,
                               caps)
        for r in range(R):
            assert torch.equal(regions_s.region(r), regions_w.region(r)), f"region {r}"
        assert np.array_equal(y_s, y_w), "y"
        ref = h.oracle_chain(cfg, inp, caps=caps)
        h.check_regions(None, regions_s, ref["regs"])
        ok, msg = h.combine_close(y_s, ref["y"])
        assert ok, msg
        h.log(f"[no-alloc] call {call} ok ({msg})")
