"""Two batches on two streams at once, each with its own workspace.

Under the default split, dispatch and combine hand parts out at run time
from ticket counters in the caller's workspace, so one workspace must not
serve two calls that run at the same time.  Separate workspaces are
independent: two batches, each with its own layout, regions and output,
launched back to back on two streams (layout, dispatch, expert and combine
of both in flight together; both layouts take the one-launch form with its
grid barrier) must each match the oracle.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import workloads as wl  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_26444_amd import moe
    moe.lib()


class _Batch:
    """One batch's device buffers and its stream."""

    def __init__(self, h, moe, cfg, stream):
        T, H, E, R, k = cfg["T"], cfg["H"], cfg["E"], cfg["R"], cfg["k"]
        self.cfg, self.stream = cfg, stream
        self.inp = wl.make_inputs(cfg)
        self.idx_d = h.to_dev(self.inp["topk_idx"].astype(np.int32))
        self.w_d = h.to_dev(self.inp["topk_w"].astype(np.float32))
        self.x_d = h.to_dev(h.u8_rows(self.inp["x"]))
        self.lay = moe.Layout(T, k, E, R)
        torch.cuda.synchronize()       # inputs were copied on the default stream
        self.lay.run(self.idx_d, stream)
        stream.synchronize()
        self.caps = self.lay.rank_count.cpu().numpy().astype(np.int32) + 1
        rows = [int(c) for c in self.caps]
        self.regions = moe.Regions(rows, wl.row_bytes(cfg), guard_bytes=h.GUARD,
                                   fill=h.SENTINEL)
        self.eregions = moe.Regions(rows, 2 * H, guard_bytes=h.GUARD, fill=h.SENTINEL)
        self.cap_d = h.to_dev(self.caps)
        self.y = torch.full((T, H), 0x5A5A, dtype=torch.int16, device="cuda")
        torch.cuda.synchronize()

    def layout(self, moe):
        self.lay.run(self.idx_d, self.stream)

    def dispatch(self, moe):
        c = self.cfg
        moe.moe_dispatch(self.x_d, None, moe.MOE_DTYPE_BF16, c["H"], c["E"], c["R"],
                         self.idx_d, self.lay.pos, self.lay.rank_offset, self.regions.table,
                         None, self.cap_d, self.lay.workspace, self.lay.status,
                         stream=self.stream)

    def expert(self, moe):
        c = self.cfg
        moe.moe_expert_scale(self.regions.table, None, moe.MOE_DTYPE_BF16, c["H"], c["E"],
                             c["R"], False, self.lay.expert_offset, self.lay.rank_offset,
                             self.cap_d, self.eregions.table, c["T"] * c["k"],
                             stream=self.stream)

    def combine(self, moe):
        c = self.cfg
        moe.moe_combine(self.eregions.table, self.w_d, c["H"], c["E"], c["R"], self.idx_d,
                        self.lay.pos, self.lay.rank_offset, self.cap_d, self.y,
                        self.lay.workspace, self.lay.status, stream=self.stream)


def test_two_streams_two_workspaces_match_oracle():
    import gpu_harness as h
    from paper_2607_26444_amd import moe
    # A: parts of >= 128 KiB, so both dispatch and combine claim every part
    # after the first; B: smaller parts, dispatch claims its second half.
    cfg_a = wl.custom(12288, 7168, 256, 64, 8, zipf_s=1.2, seed=21, name="streams_a")
    cfg_b = wl.custom(4096, 4096, 128, 32, 8, seed=22, name="streams_b")
    s_a, s_b = torch.cuda.Stream(), torch.cuda.Stream()
    a = _Batch(h, moe, cfg_a, s_a)
    b = _Batch(h, moe, cfg_b, s_b)
    h.log("[streams] launching both batches back to back")
    for _ in range(2):      # twice: the second round relies on the ticket reset
        for bt in (a, b):
            bt.regions.buf.fill_(h.SENTINEL)
            bt.y.fill_(0x5A5A)
        torch.cuda.synchronize()
        # both layouts run as one launch with a grid barrier (48 and 16
        # chunks), at the same time, each on its own workspace
        for op in ("layout", "dispatch", "expert", "combine"):
            for bt in (a, b):
                getattr(bt, op)(moe)
        torch.cuda.synchronize()
        for bt in (a, b):
            h.check_tickets_zero(bt.lay.workspace, bt.cfg["name"])
    for bt in (a, b):
        ref = h.oracle_chain(bt.cfg, bt.inp, caps=bt.caps)
        h.check_regions(None, bt.regions, ref["regs"])
        written = np.minimum(ref["layout"]["rank_count"], bt.caps)
        h.check_regions(None, bt.eregions,
                        [e.view(np.uint8).reshape(e.shape[0], 2 * e.shape[1])
                         for e in ref["ey"]], written)
        y = bt.y.cpu().numpy().view(np.uint16)
        ok, msg = h.combine_close(y, ref["y"])
        assert ok, (bt.cfg["name"], msg)
        assert int(bt.lay.status.item()) == 0
        h.log(f"[streams] {bt.cfg['name']} ok ({msg})")
