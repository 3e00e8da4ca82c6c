"""GPU parity of the layout's three launch forms, and of the fused form's
grid barrier.

moe_layout runs as one workgroup (T <= 256), as one launch whose
workgroups meet at a grid barrier (one 256-token chunk per workgroup, at
most 128 chunks), or as a count launch followed by a place launch (larger
grids).  Every form must give the oracle's layout and plan bit for bit.
The fused form keeps a generation word in the workspace (after the work
tickets) that every fused call advances; the tests read it to tell which
form ran, and check that a workspace full of leftovers -- zeros, all ones,
an increasing int64 sequence, or another batch's workspace -- never lets
the barrier pass early, including when the layout is replayed from a
captured graph with new routing between replays.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import workloads as wl  # noqa: E402

pytestmark = pytest.mark.gpu

PLAN_PARTS = 12288
# The generation word sits in the last 128 bytes of the 8 KiB ticket block,
# which follows the plan bound[PLAN_PARTS + 1] padded to 256 bytes (internal
# layout).
GEN_OFFSET = ((PLAN_PARTS + 1) * 4 + 255) // 256 * 256 + 8192 - 128


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_26444_amd import moe
    moe.lib()


def _form(T, E):
    """Launch form the library picks for (T, E) on a GPU that keeps 128
    workgroups resident: 'single', 'fused' or 'two'."""
    nc_max = 1 if E >= 32768 else 32768 // E
    per = -(-T // (256 * nc_max))
    chunk = 256 * max(1, per)
    nc = max(1, -(-T // chunk))
    if nc == 1 and T <= 256:
        return "single"
    return "fused" if chunk == 256 and 1 < nc <= 128 else "two"


def _gen(lay):
    torch.cuda.synchronize()
    return int(lay.workspace[GEN_OFFSET:GEN_OFFSET + 8].view(torch.int64).item())


def _routing(T, k, E, seed, zipf=0.0, mask=0.0):
    idx, _ = wl.make_routing(wl.custom(T, 16, E, 1, k, zipf_s=zipf, seed=seed))
    if mask:
        idx = wl.mask_slots(idx, mask, seed=seed)
    return np.ascontiguousarray(idx.astype(np.int32))


def _check(lay, idx, E, R, capacity=None, what=""):
    torch.cuda.synchronize()
    T, k = idx.shape
    ref = oracle.layout(idx, E, R) if capacity is None else \
        oracle.layout_fixed(idx, E, R, capacity)
    nrows = T * k if capacity is None else E * capacity
    got = dict(expert_count=lay.expert_count.cpu().numpy(),
               expert_offset=lay.expert_offset.cpu().numpy(),
               rank_count=lay.rank_count.cpu().numpy(),
               rank_offset=lay.rank_offset.cpu().numpy(),
               pos=lay.pos.cpu().numpy()[:T * k], row_src=lay.row_src.cpu().numpy()[:nrows])
    for key, v in got.items():
        assert np.array_equal(v, ref[key]), (what, key)
    plan = lay.plan().cpu().numpy()
    assert np.array_equal(plan, oracle.plan(ref["pos"], T, k, PLAN_PARTS)), (what, "plan")
    st = int(lay.status.item())
    assert st == ref["status"], (what, st, ref["status"])


@pytest.mark.parametrize("T,E,R,k,zipf,mask", [
    (257, 256, 64, 8, 0.0, 0.0),      # fused, 2 chunks
    (4096, 256, 64, 8, 0.0, 0.0),     # fused, decode-sized (16 chunks)
    (8192, 256, 64, 8, 1.2, 0.0),     # fused, 32 chunks, Zipf
    (16384, 256, 64, 8, 1.2, 0.0),    # fused, 64 chunks, Zipf
    (16385, 256, 64, 8, 0.0, 0.1),    # fused, 65 chunks (the last one a single token)
    (32768, 256, 64, 8, 0.0, 0.0),    # fused, 128 chunks (the most)
    (32768, 128, 32, 8, 1.5, 0.0),    # fused, 128 chunks, E = 128, Zipf
    (3000, 1, 1, 1, 0.0, 0.0),        # fused, one expert
    (5000, 1024, 64, 32, 0.0, 0.5),   # fused, widest slots and most experts
    (33024, 128, 32, 8, 0.0, 0.1),    # two launches: 129 chunks
    (65536, 16, 4, 2, 1.2, 0.0),      # two launches: 256 chunks
    (40000, 256, 64, 8, 1.2, 0.0),    # two launches: 512-token chunks
    (9000, 1024, 64, 8, 0.0, 0.1),    # two launches: 512-token chunks, E = 1024
    (200, 64, 16, 4, 0.0, 0.1),       # one workgroup
    (128, 16, 4, 2, 0.0, 0.0),        # one workgroup, the tiny workload's shape
    (1, 16, 4, 2, 0.0, 0.0),          # one token owns every part: plan written part-major
    (5, 256, 64, 8, 0.0, 0.0),        # a few tokens: plan written part-major
    (33, 64, 16, 8, 0.0, 0.5),        # part-major with unused slots
    (4096, 16, 4, 2, 0.0, 0.0),       # fused; cost total T*(1+k) equals the plan's parts
    (8192, 16, 4, 2, 0.0, 0.0),       # fused, 32 chunks; cost total is twice the plan's parts
])
def test_layout_forms_match_oracle(T, E, R, k, zipf, mask):
    from paper_2607_26444_amd import moe
    idx = _routing(T, k, E, seed=T + E, zipf=zipf, mask=mask)
    lay = moe.Layout(T, k, E, R)
    lay.workspace.fill_(0x3C)
    g0 = _gen(lay)
    lay.run(torch.from_numpy(idx).cuda())
    _check(lay, idx, E, R, what=f"T={T} E={E}")
    advanced = _gen(lay) != g0
    assert advanced == (_form(T, E) == "fused"), (T, E, _form(T, E))


@pytest.mark.parametrize("T,E,R,k,C", [(4096, 256, 64, 8, 160), (40000, 256, 64, 8, 1400),
                                       (1000, 16, 4, 4, 200),
                                       (32768, 256, 64, 8, 900)])   # one launch, 128 chunks
def test_fixed_capacity_forms_match_oracle(T, E, R, k, C):
    from paper_2607_26444_amd import moe
    idx = _routing(T, k, E, seed=T + C, zipf=1.2)
    lay = moe.Layout(T, k, E, R, capacity=C)
    lay.run(torch.from_numpy(idx).cuda())
    _check(lay, idx, E, R, capacity=C, what=f"fixed T={T} C={C}")


@pytest.mark.parametrize("T", [8192, 32768])
@pytest.mark.parametrize("fill", ["zeros", "ones", "arange", "other_batch"])
def test_fused_barrier_with_leftover_workspace(fill, T):
    """A workspace holding leftovers must not let the barrier pass before
    every chunk has published: a count row read too early would come from
    the leftovers (or an earlier batch) and misplace rows.  32 and 128
    workgroups (the most the one-launch form takes)."""
    from paper_2607_26444_amd import moe
    E, R, k = 256, 64, 8
    assert _form(T, E) == "fused"
    a = _routing(T, k, E, seed=1, zipf=1.2)
    b = _routing(T, k, E, seed=2)
    lay = moe.Layout(T, k, E, R)
    ws = lay.workspace
    if fill == "zeros":
        ws.zero_()
    elif fill == "ones":
        ws.fill_(0xFF)
    elif fill == "arange":
        n = ws.numel() // 8
        ws[:n * 8].view(torch.int64).copy_(torch.arange(n, dtype=torch.int64, device="cuda"))
    else:   # another batch's layout left its counts, flags and generation here
        lay.run(torch.from_numpy(a).cuda())
        torch.cuda.synchronize()
    lay.run(torch.from_numpy(b).cuda())
    _check(lay, b, E, R, what=fill)


def test_fused_layout_many_calls_on_one_workspace():
    """Back-to-back calls alternating two routings on one workspace: every
    call advances the generation and matches the oracle."""
    from paper_2607_26444_amd import moe
    T, E, R, k = 4096, 256, 64, 8
    routings = [_routing(T, k, E, seed=s, zipf=z) for s, z in ((11, 0.0), (12, 1.2))]
    dev = [torch.from_numpy(r).cuda() for r in routings]
    lay = moe.Layout(T, k, E, R)
    seen = {_gen(lay)}
    for i in range(12):
        lay.run(dev[i % 2])
        if i % 3 == 2:   # check some calls after several back-to-back launches
            _check(lay, routings[i % 2], E, R, what=f"call {i}")
        g = _gen(lay)
        assert g not in seen, i
        seen.add(g)


def test_fused_layout_replayed_from_a_graph_with_new_routing():
    """The fused layout captured in a graph: each replay, after new routing
    is copied into the captured input buffer, advances the generation on the
    device and matches the oracle for that routing."""
    from paper_2607_26444_amd import moe
    T, E, R, k = 6000, 128, 32, 8
    assert _form(T, E) == "fused"
    routings = [_routing(T, k, E, seed=20 + i, zipf=1.5 if i % 2 else 0.0) for i in range(4)]
    idx_d = torch.from_numpy(routings[0]).cuda()
    lay = moe.Layout(T, k, E, R)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        lay.run(idx_d)   # warm the occupancy query outside capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lay.run(idx_d)
    seen = {_gen(lay)}
    for i in range(8):
        r = routings[(i + 1) % len(routings)]
        idx_d.copy_(torch.from_numpy(r).cuda())
        lay.pos.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        _check(lay, r, E, R, what=f"replay {i}")
        gen = _gen(lay)
        assert gen not in seen, i
        seen.add(gen)


@pytest.mark.parametrize("T,E,R,k", [(4096, 256, 64, 8), (200, 64, 16, 4), (3000, 64, 16, 16)])
def test_layout_with_index_rows_off_16_byte_alignment(T, E, R, k):
    """Indices that start 4 bytes past a 16-byte boundary: the layout reads
    them one slot at a time instead of as 16-byte rows, with the same
    result."""
    from paper_2607_26444_amd import moe
    idx = _routing(T, k, E, seed=T + k, zipf=1.2)
    buf = torch.zeros(T * k + 4, dtype=torch.int32, device="cuda")
    view = buf[1:1 + T * k].view(T, k)
    assert view.data_ptr() % 16 == 4
    view.copy_(torch.from_numpy(idx).cuda())
    lay = moe.Layout(T, k, E, R)
    lay.run(view)
    _check(lay, idx, E, R, what=f"offset T={T} k={k}")


_TIME_OUT_CHILD = r'''
import sys
import numpy as np
import torch
import gpu_harness as h
import workloads as wl
from paper_2607_26444_amd import moe

T, H, E, R, k = 32768, 512, 256, 64, 8      # 128 chunks: the one-launch form
CHUNK = 256
cfg = wl.custom(T, H, E, R, k, seed=77)
inp = wl.make_inputs(cfg)
ref = h.oracle_chain(cfg, inp)
lay_ref = ref["layout"]
rows = [max(1, int(c)) for c in lay_ref["rank_count"]]
rb = 2 * H
x_d = h.to_dev(h.u8_rows(inp["x"]))
idx_d = h.to_dev(inp["topk_idx"])
w_d = h.to_dev(inp["topk_w"])
lay = moe.Layout(T, k, E, R)
regions = moe.Regions(rows, rb, guard_bytes=h.GUARD, fill=h.SENTINEL)
eregions = moe.Regions(rows, rb, guard_bytes=h.GUARD, fill=h.SENTINEL)
for r in range(R):
    n = int(lay_ref["rank_count"][r])
    if n:
        eregions.region(r)[:n].copy_(h.to_dev(ref["ey"][r].view(np.uint8).reshape(n, rb)))
cap_d = h.to_dev(np.asarray(rows, dtype=np.int32))
# rank offsets as a previous call with this routing leaves them: the first
# workgroup writes them, and may give up waiting before it does
lay.rank_offset.copy_(h.to_dev(lay_ref["rank_offset"].astype(np.int32)))
pos_ref = lay_ref["pos"].reshape(-1, CHUNK * k)
y_ref = ref["y"].reshape(T, H)
late_calls = 0
for call in range(6):
    print("[child] call", call, flush=True)
    regions.buf.fill_(h.SENTINEL)
    y = torch.full((T, H), 0x5A5A, dtype=torch.int16, device="cuda")
    lay.status.zero_()
    lay.run(idx_d)
    moe.moe_dispatch(x_d, None, moe.MOE_DTYPE_BF16, H, E, R, idx_d, lay.pos, lay.rank_offset,
                     regions.table, None, cap_d, lay.workspace, lay.status)
    moe.moe_combine(eregions.table, w_d, H, E, R, idx_d, lay.pos, lay.rank_offset, cap_d, y,
                    lay.workspace, lay.status)
    torch.cuda.synchronize()
    st = int(lay.status.item())
    pos = lay.pos.cpu().numpy()[:T * k].reshape(-1, CHUNK * k)
    late = np.array([bool((p == -1).all()) for p in pos])
    for c in range(len(pos)):
        assert late[c] or np.array_equal(pos[c], pos_ref[c]), ("chunk misplaced", call, c)
    if st & moe.MOE_STATUS_LAYOUT_SYNC:
        late_calls += 1
    else:
        assert not late.any(), ("chunks unrouted without the status bit", call)
    # regions: every row is untouched or the oracle's; nothing outside them
    buf = regions.buf.cpu().numpy()
    inside = np.zeros(buf.shape[0], bool)
    for r, off in enumerate(regions.offsets):
        got = buf[off: off + rows[r] * rb].reshape(rows[r], rb)
        want = ref["regs"][r]
        n = want.shape[0]
        untouched = (got == h.SENTINEL).all(1)
        assert np.all(untouched[n:]), ("row past the routed rows written", call, r)
        assert np.all(untouched[:n] | (got[:n] == want).all(1)), ("wrong row", call, r)
        inside[off: off + rows[r] * rb] = True
    assert np.all(buf[~inside] == h.SENTINEL), ("bytes outside the regions", call)
    # y: each row untouched, zero (a token left unrouted) or the oracle's
    yy = y.cpu().numpy().view(np.uint16)
    untouched = (yy == 0x5A5A).all(1)
    zero = (yy == 0).all(1)
    rest = ~(untouched | zero)
    assert not np.any(zero & ~np.repeat(late, CHUNK)), ("zero row of a placed chunk", call)
    ok, msg = h.combine_close(yy[rest], y_ref[rest])
    assert ok, (call, msg)
    print("[child] call", call, "status", st, "unrouted chunks", int(late.sum()), flush=True)
print("ok", late_calls, flush=True)
'''


def test_barrier_time_out_keeps_every_write_in_bounds():
    """The barrier's time limit forced to zero from the host
    (MOE_LAYOUT_SYNC_LIMIT_US=0, in a child process, so that the limit holds
    from the library's first launch): a workgroup that does not see every
    flag at its first look gives up.  Its chunk's slots come back unrouted,
    every other chunk's positions equal the oracle's, the status word says
    MOE_STATUS_LAYOUT_SYNC, and dispatch and combine, run on whatever the
    layout left (parts of the plan unwritten), write only rows the oracle
    has and nothing outside their buffers."""
    import os
    import subprocess
    import sys
    here = os.path.dirname(os.path.abspath(__file__))
    env = dict(os.environ, MOE_LAYOUT_SYNC_LIMIT_US="0",
               PYTHONPATH=os.pathsep.join([os.path.dirname(here), here,
                                           os.environ.get("PYTHONPATH", "")]))
    r = subprocess.run([sys.executable, "-u", "-c", _TIME_OUT_CHILD], env=env,
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    last = r.stdout.strip().splitlines()[-1]
    assert last.startswith("ok"), r.stdout[-3000:]
    print(r.stdout[-2000:])
