"""Benchmark of the MoE dispatch/combine hot path on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                [--no-cpu-baseline] [--ablation]

One step = one pass of the whole path on one batch already resident in HBM:
moe_layout (histograms, scans, placement, partition plan) -> moe_dispatch
(rows into R emulated rank regions) -> moe_combine (top-k weighted gather).
The stand-in expert between dispatch and combine is run once before timing
(it is not part of the operator); combine reads its outputs every step.

Prints one JSON line.  `value` is dispatch+combine algorithmic bytes per
second of whole-step time (the layout's time is included, its bytes are
not credited).  Algorithmic bytes: dispatch reads x once and writes every
routed row plus 4 bytes of pos per slot; combine reads every routed row
plus 8 bytes (weight, pos) per slot and writes y.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
# Per-phase timing events go on every EVENT_EVERY-th timed step (see main).
EVENT_EVERY = 4


def sampled_steps(steps: int, every: int) -> list:
    """Timed steps that carry per-phase events: 0, every, 2*every, ..."""
    return list(range(0, steps, max(1, every)))


def _num(v, nd):
    return None if v != v else round(v, nd)   # NaN -> null


_HIP = None
_HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000   # hip_runtime_api.h


def _hip():
    """The HIP runtime torch has loaded (the same instance libmoe uses)."""
    global _HIP
    if _HIP is None:
        import ctypes
        import torch
        torch.cuda.init()
        paths = {line.split()[-1] for line in open("/proc/self/maps")
                 if "libamdhip64" in line and line.split()[-1].startswith("/")}
        if len(paths) != 1:
            raise RuntimeError(f"expected one loaded HIP runtime, found {sorted(paths)}")
        L = ctypes.CDLL(paths.pop())
        vp = ctypes.c_void_p
        L.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
        L.hipEventRecord.argtypes = [vp, vp]
        L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), vp, vp]
        L.hipEventDestroy.argtypes = [vp]
        for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipEventElapsedTime",
                  "hipEventDestroy"):
            getattr(L, f).restype = ctypes.c_int
        _HIP = L
    return _HIP


class Event:
    """A timing event recorded on a stream, with torch's Event interface
    (record, elapsed_time in ms).  It is a HIP event created with
    hipEventDisableSystemFence: torch's events perform a system-scope fence
    at every record, a cache write-back and invalidate that the next kernel
    then pays for, and that no real pipeline runs between these kernels
    (measured on MI355X: 12-13 us more per step with four torch events per
    step)."""

    def __init__(self):
        import ctypes
        self._ct = ctypes
        self._hip = _hip()
        self._e = ctypes.c_void_p()
        rc = self._hip.hipEventCreateWithFlags(ctypes.byref(self._e),
                                               _HIP_EVENT_DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags failed: {rc}")

    def record(self, stream=None):
        import torch
        s = stream if stream is not None else torch.cuda.current_stream()
        rc = self._hip.hipEventRecord(self._e, self._ct.c_void_p(s.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed: {rc}")

    def elapsed_time(self, end: "Event") -> float:
        ms = self._ct.c_float()
        rc = self._hip.hipEventElapsedTime(self._ct.byref(ms), self._e, end._e)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return ms.value

    def __del__(self):
        try:
            if self._e:
                self._hip.hipEventDestroy(self._e)
        except Exception:
            pass


def algorithmic_bytes(cfg) -> dict:
    T, H, k = cfg["T"], cfg["H"], cfg["k"]
    fp8 = cfg["payload"] == 1
    row = H * (1 if fp8 else 2) + ((H // 128) * 4 if fp8 else 0)
    n = T * k
    d_read, d_write = T * row + 4 * n, n * row
    c_read, c_write = n * 2 * H + 8 * n, T * 2 * H
    return dict(dispatch=d_read + d_write, combine=c_read + c_write, row=row, n=n,
                dispatch_read=d_read, dispatch_write=d_write,
                combine_read=c_read, combine_write=c_write)


def stream_ceiling(read_bytes, write_bytes, read_GBps, write_GBps):
    """GB/s of a kernel that reads read_bytes and writes write_bytes if its
    reads ran at the pure-read rate and its writes at the pure-write rate,
    one after the other.  Mixing the two in one stream only adds read/write
    turnarounds, so this bounds what a mixed kernel can reach."""
    t = read_bytes / read_GBps + write_bytes / write_GBps
    return (read_bytes + write_bytes) / t if t > 0 else float("nan")


def measure_stream_legs(dev, stream, read_bytes, write_bytes, reps=10):
    """Pure-write and pure-read rates on this GPU, built from torch ops (no
    kernel of this library): fill_ of a buffer of write_bytes, and reductions
    over a buffer of read_bytes -- a float32 sum along rows of 4096, a bf16
    matrix-vector product over rows of 4096 and a whole-buffer float32 sum
    (the fastest counts; on MI355X the row sum reads ~6.4 TB/s, the
    whole-buffer sum ~4 TB/s).  GB/s of the bytes each op moves."""
    import torch
    out = {}
    buf = torch.empty(max(1 << 20, write_bytes // 16 * 16), dtype=torch.uint8, device=dev)
    for i in range(3):
        buf.fill_(i)
    e0, e1 = Event(), Event()
    e0.record(stream)
    for i in range(reps):
        buf.fill_(i & 0xFF)
    e1.record(stream)
    torch.cuda.synchronize()
    out["write_GBps"] = buf.numel() * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    out["write_buffer_bytes"] = buf.numel()
    del buf
    buf = torch.zeros(max(1 << 20, read_bytes // 16 * 16), dtype=torch.uint8, device=dev)
    rates = {}
    buf = buf[: buf.numel() // (1 << 14) * (1 << 14)]   # whole rows of 4096 float32
    vec = torch.ones(4096, dtype=torch.bfloat16, device=dev)
    for name, op in (("rowsum_f32", lambda b: b.view(torch.float32).view(-1, 4096).sum(dim=1)),
                     ("mv_bf16", lambda b: torch.mv(b.view(torch.bfloat16).view(-1, 4096), vec)),
                     ("sum_f32", lambda b: b.view(torch.float32).sum())):
        for _ in range(3):
            op(buf)
        e0.record(stream)
        for _ in range(reps):
            op(buf)
        e1.record(stream)
        torch.cuda.synchronize()
        rates[name] = buf.numel() * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
    out["read_op"] = max(rates, key=rates.get)
    out["read_GBps"] = rates[out["read_op"]]
    out["read_rates_GBps"] = {n: round(v, 1) for n, v in rates.items()}
    out["read_buffer_bytes"] = buf.numel()
    del buf
    return out


def kernel_source_hash(kernel: str) -> str:
    """Hash of the device code of one kernel: its source file and the shared
    device header."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_26444_amd", "csrc")
    for f in (f"{kernel}.hip", "moe_internal.h"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def read_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            a, b = line.split(":", 1)
            kv[a.strip()] = b.strip()
    if kv.get("source_hash") != kernel_source_hash(kernel):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(cfg, inp, budget_s=20.0, max_reps=5, capacity=None):
    """The CPU oracle (single-threaded) on the same workload: layout (the
    fixed-capacity one when `capacity` is set), dispatch and combine, timed
    on this host.  Its combine reads the dispatched rows directly (identity
    expert); the cost does not depend on the values."""
    import oracle
    E, R, H = cfg["E"], cfg["R"], cfg["H"]
    fp8 = cfg["payload"] == 1
    x_rows = np.ascontiguousarray(inp["x"]).view(np.uint8).reshape(cfg["T"], -1)
    xs_rows = (np.ascontiguousarray(inp["x_scales"]).view(np.uint8).reshape(cfg["T"], -1)
               if fp8 else None)
    times = []
    t_start = time.perf_counter()
    for _ in range(max_reps):
        t0 = time.perf_counter()
        if capacity is None:
            lay = oracle.layout(inp["topk_idx"], E, R)
            caps = lay["rank_count"]
        else:
            lay = oracle.layout_fixed(inp["topk_idx"], E, R, capacity)
            caps = np.full(R, (E // R) * capacity, np.int32)
        t1 = time.perf_counter()
        regs, _, _ = oracle.dispatch(x_rows, xs_rows, inp["topk_idx"], lay["pos"],
                                     lay["rank_offset"], E, R, caps)
        t2 = time.perf_counter()
        if fp8:
            ey = [np.zeros((r.shape[0], H), np.uint16) for r in regs]
        else:
            ey = [r.view(np.uint16).reshape(r.shape[0], H) for r in regs]
        t3 = time.perf_counter()
        oracle.combine(ey, inp["topk_w"], inp["topk_idx"], lay["pos"], lay["rank_offset"],
                       caps, E, R, H)
        t4 = time.perf_counter()
        times.append((t1 - t0) + (t2 - t1) + (t4 - t3))
        del regs, ey
        if time.perf_counter() - t_start > budget_s:
            break
    return float(np.median(times)), len(times)


def cpu_baseline_dedup(cfg, inp, n_tokens, budget_s=20.0, max_reps=5):
    """The CPU oracle's deduplicated chain on the first n_tokens tokens of
    the workload (both layouts, pair dispatch, expansion, partial combine,
    source sum; the expanded rows stand in for expert outputs), timed on
    this host."""
    import oracle
    E, R, H = cfg["E"], cfg["R"], cfg["H"]
    fp8 = cfg["payload"] == 1
    n = n_tokens
    idx = np.ascontiguousarray(inp["topk_idx"][:n])
    x_rows = np.ascontiguousarray(inp["x"][:n]).view(np.uint8).reshape(n, -1)
    xs_rows = (np.ascontiguousarray(inp["x_scales"][:n]).view(np.uint8).reshape(n, -1)
               if fp8 else None)
    w = np.ascontiguousarray(inp["topk_w"][:n])
    srb = xs_rows.shape[1] if fp8 else 0
    times = []
    t_start = time.perf_counter()
    for _ in range(max_reps):
        t0 = time.perf_counter()
        lay = oracle.layout(idx, E, R)
        d = oracle.layout_dedup(idx, E, R)
        dregs, dsregs, _ = oracle.dispatch_dedup(x_rows, xs_rows, idx, d["tok_pos"],
                                                 d["tok_offset"], E, R, d["tok_count"])
        regs, _, _ = oracle.expand(dregs, dsregs, srb, idx, lay["pos"], lay["rank_offset"],
                                   d["tok_pos"], d["tok_offset"], d["tok_count"], E, R,
                                   lay["rank_count"])
        t1 = time.perf_counter()
        if fp8:
            ey = [np.zeros((r.shape[0], H), np.uint16) for r in regs]
        else:
            ey = [r.view(np.uint16).reshape(r.shape[0], H) for r in regs]
        t2 = time.perf_counter()
        parts, _ = oracle.combine_local(ey, w, idx, lay["pos"], lay["rank_offset"],
                                        lay["rank_count"], d["tok_pos"], d["tok_offset"],
                                        d["tok_count"], E, R, H)
        oracle.combine_dedup(parts, idx, d["tok_pos"], d["tok_offset"], d["tok_count"], E, R,
                             H)
        t3 = time.perf_counter()
        times.append((t1 - t0) + (t3 - t2))
        del dregs, regs, ey, parts
        if time.perf_counter() - t_start > budget_s:
            break
    return float(np.median(times)), len(times)


def trace_stats(trace, khz):
    """Per-wavefront completion times from a (start, end) trace: makespan and
    the fastest-to-slowest completion gap (Section 9.6 reports this gap per
    core), relative to the earliest start."""
    t = trace.view(-1, 2).cpu().numpy().astype(np.int64)
    t = t[t[:, 0] != 0]
    t0 = t[:, 0].min()
    done = (t[:, 1] - t0) / khz * 1e3          # microseconds
    busy = (t[:, 1] - t[:, 0]) / khz * 1e3
    return dict(waves=int(len(t)), makespan_us=round(float(done.max()), 2),
                completion_gap_pct=round(100 * float((done.max() - done.min()) / done.max()), 1),
                completion_p10_us=round(float(np.percentile(done, 10)), 2),
                completion_p90_us=round(float(np.percentile(done, 90)), 2),
                busy_mean_us=round(float(busy.mean()), 2))


def hidden_copies(x_d, xs_d, n):
    """Copies of the hidden states (and fp8 scales) for the timed steps to
    cycle through, each step reading its own as each layer of a model does.
    n = 0: copies that fill 512 MiB (at most 16), so a step does not find
    its x in the 256 MB Infinity Cache, where the previous read of the same
    x would otherwise leave it (the rest of a step streams non-temporally
    past the cache)."""
    n = n if n > 0 else min(16, max(1, -(-(512 << 20) // x_d.numel())))
    return [(x_d, xs_d)] + [(x_d.clone(), None if xs_d is None else xs_d.clone())
                            for _ in range(n - 1)]


def ablation(a):
    """Dispatch under the three work splits of moe_dispatch_ex on one
    workload: kernel time (HIP events) and the per-wavefront completion trace.
    One JSON line."""
    import torch
    import workloads as wl
    from paper_2607_26444_amd import moe

    cfg = wl.get(a.workload)
    T, H, E, R, k = cfg["T"], cfg["H"], cfg["E"], cfg["R"], cfg["k"]
    fp8 = cfg["payload"] == wl.FP8_E4M3
    dtype = moe.MOE_DTYPE_FP8_E4M3 if fp8 else moe.MOE_DTYPE_BF16
    inp = wl.make_inputs(cfg)
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream()
    x_d = torch.from_numpy(np.ascontiguousarray(inp["x"]).view(np.uint8)).to(dev)
    xs_d = torch.from_numpy(inp["x_scales"]).to(dev) if fp8 else None
    xs_all = hidden_copies(x_d, xs_d, a.x_copies)
    n_calls = [0]
    idx_d = torch.from_numpy(inp["topk_idx"]).to(dev)
    lay = moe.Layout(T, k, E, R)
    lay.run(idx_d)
    torch.cuda.synchronize()
    rows = [max(1, int(c)) for c in lay.rank_count.cpu().numpy()]
    sb = wl.scale_row_bytes(cfg)
    spitch = (sb + 127) // 128 * 128
    regions = moe.Regions(rows, wl.row_bytes(cfg))
    sregions = moe.Regions(rows, spitch) if fp8 else None
    trace = torch.zeros(2 * moe.MOE_PLAN_PARTS, dtype=torch.int64, device=dev)
    khz = moe.moe_wall_clock_khz()
    out = {"metric": "dispatch work-split ablation",
           "config": {"workload": cfg["name"], "x_copies": len(xs_all)},
           "rank_rows_max_over_mean": round(max(rows) / (sum(rows) / len(rows)), 2),
           "wall_clock_khz": khz, "policies": {}}
    b = algorithmic_bytes(cfg)

    def time_dispatch(pol, waves=0):
        def run(tr=None):
            xc, xsc = xs_all[n_calls[0] % len(xs_all)]
            n_calls[0] += 1
            moe.moe_dispatch_ex(xc, xsc, dtype, H, E, R, idx_d, lay.pos, lay.rank_offset,
                                lay.row_src, regions.table,
                                sregions.table if fp8 else None, regions.cap, lay.workspace,
                                lay.status, policy=pol, trace=tr, scale_pitch=spitch,
                                waves=waves)
        for _ in range(3):
            run()
        e0, e1 = Event(), Event()
        e0.record(stream)
        for _ in range(a.steps):
            run()
        e1.record(stream)
        trace.zero_()
        run(trace)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / a.steps
        rec = dict(dispatch_us=round(us, 2), GBps=round(b["dispatch"] / (us * 1e-6) / 1e9, 1))
        rec.update(trace_stats(trace, khz))
        return rec

    for name, pol in (("balanced_push", moe.MOE_POLICY_BALANCED),
                      ("static_push", moe.MOE_POLICY_STATIC),
                      ("dynamic_push", moe.MOE_POLICY_DYNAMIC),
                      ("rows_pull", moe.MOE_POLICY_ROWS),
                      ("by_rank_pull", moe.MOE_POLICY_BY_RANK)):
        rec = time_dispatch(pol)
        out["policies"][name] = rec
        print(f"[ablation] {name}: {rec}", file=sys.stderr, flush=True)
    # wavefront-count sweep: 4 wavefronts per workgroup, so W wavefronts
    # occupy up to W/4 compute units
    out["wave_sweep"] = []
    for waves in (R, 2 * R, 4 * R, 8 * R, 16 * R):
        if moe.MOE_PLAN_PARTS % waves or waves % 4:
            continue
        rec = {"waves": waves}
        for name, pol in (("balanced_push", moe.MOE_POLICY_BALANCED),
                          ("static_push", moe.MOE_POLICY_STATIC),
                          ("by_rank_pull", moe.MOE_POLICY_BY_RANK)):
            r = time_dispatch(pol, waves)
            rec[name] = {k2: r[k2] for k2 in ("dispatch_us", "GBps", "completion_gap_pct")}
        out["wave_sweep"].append(rec)
        print(f"[ablation] sweep {rec}", file=sys.stderr, flush=True)
    # combine: static vs dynamic part assignment (expert outputs = the rows)
    w_d = torch.from_numpy(inp["topk_w"]).to(dev)
    if not fp8:
        y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        out["combine"] = {}
        for name, pol in (("balanced", moe.MOE_POLICY_BALANCED),
                          ("dynamic", moe.MOE_POLICY_DYNAMIC)):   # balanced = static here
            def runc(tr=None):
                moe.moe_combine_ex(regions.table, w_d, H, E, R, idx_d, lay.pos,
                                   lay.rank_offset, regions.cap, y, lay.workspace, lay.status,
                                   policy=pol, trace=tr)
            for _ in range(3):
                runc()
            e0, e1 = Event(), Event()
            e0.record(stream)
            for _ in range(a.steps):
                runc()
            e1.record(stream)
            trace.zero_()
            runc(trace)
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / a.steps
            rec = dict(combine_us=round(us, 2), GBps=round(b["combine"] / (us * 1e-6) / 1e9, 1))
            rec.update(trace_stats(trace, khz))
            out["combine"][name] = rec
            print(f"[ablation] combine {name}: {rec}", file=sys.stderr, flush=True)
    st = int(lay.status.item())
    out["status"] = st
    print(json.dumps(out), flush=True)
    return 0 if st == 0 else 1


def dedup_bench(a):
    """The per-peer deduplicated path on one workload: per-kernel time (HIP
    events on the launch stream) and GB/s of each kernel's algorithmic
    bytes, the pair-row fraction (bytes that would cross to peers, relative
    to one row per routed slot) and the per-slot step beside it.  One JSON
    line."""
    import torch
    import workloads as wl
    from paper_2607_26444_amd import moe

    cfg = wl.get(a.workload)
    T, H, E, R, k = cfg["T"], cfg["H"], cfg["E"], cfg["R"], cfg["k"]
    fp8 = cfg["payload"] == wl.FP8_E4M3
    dtype = moe.MOE_DTYPE_FP8_E4M3 if fp8 else moe.MOE_DTYPE_BF16
    print(f"[dedup] workload {cfg['name']}: generating inputs", file=sys.stderr, flush=True)
    inp = wl.make_inputs(cfg)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    x_d = torch.from_numpy(np.ascontiguousarray(inp["x"]).view(np.uint8)).to(dev)
    xs_d = torch.from_numpy(inp["x_scales"]).to(dev) if fp8 else None
    xs_all = hidden_copies(x_d, xs_d, a.x_copies)
    cur = [0]
    idx_d = torch.from_numpy(inp["topk_idx"]).to(dev)
    w_d = torch.from_numpy(inp["topk_w"]).to(dev)
    lay = moe.Layout(T, k, E, R)
    dl = moe.DedupLayout(T, k, E, R)
    lay.run(idx_d)
    dl.run(idx_d)
    torch.cuda.synchronize()
    rows = [max(1, int(c)) for c in lay.rank_count.cpu().numpy()]
    prow = [max(1, int(c)) for c in dl.tok_count.cpu().numpy()]
    n_slots, n_pairs = int(lay.rank_offset[-1].item()), int(dl.tok_offset[-1].item())
    rb, sb = wl.row_bytes(cfg), wl.scale_row_bytes(cfg)
    spitch = (sb + 127) // 128 * 128
    dreg = moe.Regions(prow, rb)
    dsreg = moe.Regions(prow, spitch) if fp8 else None
    reg = moe.Regions(rows, rb)
    sreg = moe.Regions(rows, spitch) if fp8 else None
    reg_ps = moe.Regions(rows, rb)           # the per-slot reference dispatch's own
    sreg_ps = moe.Regions(rows, spitch) if fp8 else None
    ereg = moe.Regions(rows, 2 * H)
    preg = moe.Regions(prow, 2 * H)
    y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)

    ops = {
        "layout": lambda: lay.run(idx_d),
        "layout_dedup": lambda: dl.run(idx_d),
        "dispatch_dedup": lambda: moe.moe_dispatch_dedup(
            *xs_all[cur[0]], dtype, H, E, R, idx_d, dl.tok_pos, dl.tok_offset, dreg.table,
            dsreg.table if fp8 else None, dreg.cap, dl.workspace, status, scale_pitch=spitch),
        "expand": lambda: moe.moe_expand(
            dreg.table, dsreg.table if fp8 else None, dtype, H, E, R, idx_d, lay.pos,
            lay.rank_offset, dl.tok_pos, dl.tok_offset, dreg.cap, reg.table,
            sreg.table if fp8 else None, reg.cap, lay.workspace, status, scale_pitch=spitch),
        "combine_local": lambda: moe.moe_combine_local(
            ereg.table, w_d, H, E, R, idx_d, lay.pos, lay.rank_offset, ereg.cap, dl.tok_pos,
            dl.tok_offset, preg.cap, preg.table, lay.workspace, status),
        "combine_dedup": lambda: moe.moe_combine_dedup(
            preg.table, H, E, R, idx_d, dl.tok_pos, dl.tok_offset, preg.cap, y, dl.workspace,
            status),
        "dispatch": lambda: moe.moe_dispatch(
            *xs_all[cur[0]], dtype, H, E, R, idx_d, lay.pos, lay.rank_offset, reg_ps.table,
            sreg_ps.table if fp8 else None, reg_ps.cap, lay.workspace, status,
            scale_pitch=spitch),
        "combine": lambda: moe.moe_combine(
            ereg.table, w_d, H, E, R, idx_d, lay.pos, lay.rank_offset, ereg.cap, y,
            lay.workspace, status),
    }
    ops["dispatch"]()
    moe.moe_expert_scale(reg_ps.table, sreg_ps.table if fp8 else None, dtype, H, E, R,
                         cfg["expert"] == "identity", lay.expert_offset, lay.rank_offset,
                         reg_ps.cap, ereg.table, sum(rows), scale_pitch=spitch)
    torch.cuda.synchronize()
    names = list(ops)
    # Each path is timed in steps of its own, as a layer runs one of them: the
    # per-slot dispatch stores rows of 8 KiB or less with ordinary stores,
    # and their write-back, interleaved with the per-peer chain, made the
    # expansion 8-13% slower at the large and fp8 workloads.
    phases = (["layout", "layout_dedup", "dispatch_dedup", "expand", "combine_local",
               "combine_dedup"], ["dispatch", "combine"])
    ev = {n: [(Event(), Event())
              for _ in range(a.steps)] for n in names}
    for phase in phases:
        for i in range(a.warmup):
            cur[0] = i % len(xs_all)
            for n in phase:
                ops[n]()
        torch.cuda.synchronize()
        for s_ in range(a.steps):
            cur[0] = s_ % len(xs_all)
            for n in phase:
                ev[n][s_][0].record(stream)
                ops[n]()
                ev[n][s_][1].record(stream)
        torch.cuda.synchronize()
    st = int(status.item()) | int(lay.status.item()) | int(dl.status.item())
    us = {n: float(np.mean([e0.elapsed_time(e1) for e0, e1 in ev[n]])) * 1e3 for n in names}
    row = rb + sb                        # a row and its scales (fp8)
    alg = {
        "dispatch_dedup": T * row + n_pairs * row + 4 * T * k,
        "expand": n_pairs * row + n_slots * row + 8 * T * k,
        "combine_local": n_slots * 2 * H + n_pairs * 2 * H + 12 * T * k,
        "combine_dedup": n_pairs * 2 * H + T * 2 * H + 4 * T * k,
        "dispatch": T * row + n_slots * row + 4 * T * k,
        "combine": n_slots * 2 * H + T * 2 * H + 8 * T * k,
    }
    kern = {n: {"us": round(us[n], 2)} for n in names}
    for n, b in alg.items():
        kern[n].update(bytes=int(b), GBps=round(b / (us[n] * 1e-6) / 1e9, 1),
                       frac=round(b / (us[n] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4))
    dedup_step = sum(us[n] for n in ("layout", "layout_dedup", "dispatch_dedup", "expand",
                                     "combine_local", "combine_dedup"))
    slot_step = sum(us[n] for n in ("layout", "dispatch", "combine"))
    out = {
        "metric": "per-peer deduplicated dispatch/combine: per-kernel HBM GB/s",
        "config": {"workload": cfg["name"], "T": T, "H": H, "E": E, "R": R, "k": k,
                   "payload": "fp8_e4m3" if fp8 else "bf16", "x_copies": len(xs_all)},
        "steps": a.steps, "warmup": a.warmup,
        "slots": n_slots, "pair_rows": n_pairs,
        "pair_row_fraction": round(n_pairs / max(1, n_slots), 4),
        "peer_bytes_dispatch": {"per_slot": n_slots * row, "dedup": n_pairs * row},
        "peer_bytes_combine": {"per_slot": n_slots * 2 * H, "dedup": n_pairs * 2 * H},
        "kernels": kern,
        "dedup_step_us": round(dedup_step, 2),
        "per_slot_step_us": round(slot_step, 2),
        "status": st,
        "cpu_baseline": None,
    }
    if not a.no_cpu_baseline:
        print("[dedup] timing the CPU oracle", file=sys.stderr, flush=True)
        n_s = min(T, 2048)   # a bounded sample: the first n_s tokens
        cpu_s, reps = cpu_baseline_dedup(cfg, inp, n_s)
        full_us = cpu_s * 1e6 * T / n_s
        out["cpu_baseline"] = {
            "step_us": round(full_us, 1), "unit": "us per full step (scaled)", "cores": 1,
            "kind": "oracle",
            "sample": f"first {n_s} of {T} tokens (both layouts, pair dispatch, expansion, "
                      f"partial combine, source sum), median of {reps} run(s), {cpu_s:.2f} s "
                      f"each, scaled by {T}/{n_s}; 1 thread, host CPU: {cpu_model()}",
            "gpu_speedup": round(full_us / dedup_step, 1), "host_nproc": os.cpu_count()}
    print(json.dumps(out), flush=True)
    return 0 if st == 0 else 1


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 100; 1000 for the tiny workload)")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="prefill")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--ablation", action="store_true",
                    help="instead of the step benchmark: dispatch under each work split")
    ap.add_argument("--ll", type=float, default=None, metavar="F",
                    help="fixed-capacity layout with windows of F x the mean expert load")
    ap.add_argument("--x-copies", type=int, default=0, metavar="N",
                    help="hidden-state copies the timed steps cycle through (0: enough to "
                         "fill 512 MiB, at most 16, so a step's x is not in the 256 MB "
                         "Infinity Cache; 1: every step reads the same x)")
    ap.add_argument("--cold-reps", type=int, default=20,
                    help="repetitions of the cold-cache pass (0 skips it)")
    ap.add_argument("--dedup", action="store_true",
                    help="instead of the step benchmark: the per-peer deduplicated path")
    ap.add_argument("--graph", action="store_true",
                    help="capture the steps in graphs, one step per x copy in each "
                         "(needs --ll: no host sync in a step)")
    ap.add_argument("--event-every", type=int, default=EVENT_EVERY, metavar="N",
                    help="record the per-phase timing events on every N-th timed step "
                         "(1: every step)")
    a = ap.parse_args(argv)
    if a.steps is None:
        a.steps = 1000 if a.workload in ("tiny", "tiny_t128_h256_e16_r4_k2") else 100
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU's share of the operator; runs on more than "
              "one GPU are not supported (use --gpus 1).", file=sys.stderr)
        return 2

    if a.ablation:
        return ablation(a)
    if a.dedup:
        return dedup_bench(a)

    import torch
    import workloads as wl
    from paper_2607_26444_amd import moe

    cfg = wl.get(a.workload)
    T, H, E, R, k = cfg["T"], cfg["H"], cfg["E"], cfg["R"], cfg["k"]
    fp8 = cfg["payload"] == wl.FP8_E4M3
    dtype = moe.MOE_DTYPE_FP8_E4M3 if fp8 else moe.MOE_DTYPE_BF16
    print(f"[bench] workload {cfg['name']}: generating inputs", file=sys.stderr, flush=True)
    inp = wl.make_inputs(cfg)

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    x_d = torch.from_numpy(np.ascontiguousarray(inp["x"]).view(np.uint8)).to(dev)
    xs_d = torch.from_numpy(inp["x_scales"]).to(dev) if fp8 else None
    idx_d = torch.from_numpy(inp["topk_idx"]).to(dev)
    w_d = torch.from_numpy(inp["topk_w"]).to(dev)
    xs_all = hidden_copies(x_d, xs_d, a.x_copies)
    n_x = len(xs_all)
    cur = [0]

    if a.graph and a.ll is None:
        print("--graph needs --ll (the packed layout reads counts back to size regions)",
              file=sys.stderr)
        return 2
    capacity = None if a.ll is None else max(1, int(np.ceil(a.ll * T * k / E)))
    lay = moe.Layout(T, k, E, R, capacity=capacity)
    lay.run(idx_d)
    torch.cuda.synchronize()
    if capacity is None:
        counts = lay.rank_count.cpu().numpy()
        rows = [max(1, int(c)) for c in counts]
    else:   # whole windows, sized before routing is known
        rows = [(E // R) * capacity] * R
    rb, sb = wl.row_bytes(cfg), wl.scale_row_bytes(cfg)
    spitch = (sb + 127) // 128 * 128   # scale rows on whole 128-byte lines
    regions = moe.Regions(rows, rb)
    sregions = moe.Regions(rows, spitch) if fp8 else None
    eregions = moe.Regions(rows, 2 * H)
    y = torch.empty((T, H), dtype=torch.bfloat16, device=dev)

    def dispatch():
        xc, xsc = xs_all[cur[0]]
        moe.moe_dispatch(xc, xsc, dtype, H, E, R, idx_d, lay.pos, lay.rank_offset,
                         regions.table, sregions.table if fp8 else None, regions.cap,
                         lay.workspace, lay.status, scale_pitch=spitch)

    def combine():
        moe.moe_combine(eregions.table, w_d, H, E, R, idx_d, lay.pos, lay.rank_offset,
                        eregions.cap, y, lay.workspace, lay.status)

    # stand-in expert outputs for combine (once, untimed)
    dispatch()
    moe.moe_expert_scale(regions.table, sregions.table if fp8 else None, dtype, H, E, R,
                         cfg["expert"] == "identity", lay.expert_offset, lay.rank_offset,
                         regions.cap, eregions.table, sum(rows), scale_pitch=spitch)
    torch.cuda.synchronize()

    for i in range(a.warmup):
        cur[0] = i % n_x
        lay.run(idx_d)
        dispatch()
        combine()
    torch.cuda.synchronize()
    status = int(lay.status.item())
    if status != 0:
        print(f"[bench] status word {status} after warmup", file=sys.stderr)
        if capacity is not None and status == moe.MOE_STATUS_CAPACITY:
            ti = inp["topk_idx"]
            need = np.bincount(ti[ti >= 0].ravel(), minlength=E).max() * E / (T * k)
            print(f"[bench] the fixed windows drop slots: the busiest expert needs "
                  f"--ll {need:.2f} or more", file=sys.stderr)
        return 1

    # Per-phase events on every N-th timed step (`sampled`), one per phase
    # boundary; on consecutive sampled steps the event that closes a step's
    # combine also opens the next step's layout.
    every = max(1, a.event_every)
    sampled = sampled_steps(a.steps, every)
    ev = {}
    for s in sampled:
        ev[s] = [ev[s - 1][-1] if s - 1 in ev else Event()] + [Event() for _ in range(3)]
    graph = None
    if a.graph:
        # Graphs of consecutive steps, one step per x copy in order (the last
        # replay may hold fewer): a replay's own start and end are paid once
        # per graph, not once per step.  Events stay outside the graphs,
        # around every replay.
        def capture(n):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(n):
                    cur[0] = i
                    lay.run(idx_d)
                    dispatch()
                    combine()
            return g
        gsteps = n_x
        graph = {gsteps: capture(gsteps)}
        if a.steps % gsteps:
            graph[a.steps % gsteps] = capture(a.steps % gsteps)
        torch.cuda.synchronize()
        for _ in range(3):
            for g in graph.values():
                g.replay()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        replays = [min(gsteps, a.steps - s) for s in range(0, a.steps, gsteps)]
        rev = [(Event(), Event()) for _ in replays]
    print(f"[bench] timing {a.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if graph is not None:
        for n, (e0, e1) in zip(replays, rev):
            e0.record(stream)
            graph[n].replay()
            e1.record(stream)
    for s in range(a.steps if graph is None else 0):
        cur[0] = s % n_x
        e = ev.get(s)
        if e is not None and s - 1 not in ev:
            e[0].record(stream)
        if e is not None:
            lay.run(idx_d)
            e[1].record(stream)
            dispatch()
            e[2].record(stream)
            combine()
            e[3].record(stream)
        else:
            lay.run(idx_d)
            dispatch()
            combine()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    status = int(lay.status.item())
    if status != 0:
        print(f"[bench] status word {status} after timing", file=sys.stderr)
        return 1

    # per-phase times of the sampled steps (with graphs, lay_ms holds each
    # replay's time per step)
    if graph is not None:
        sampled = list(range(0, a.steps, gsteps))
        lay_ms = np.array([e0.elapsed_time(e1) / n for n, (e0, e1) in zip(replays, rev)])
        dis_ms = com_ms = np.full(len(replays), float("nan"))
    else:
        lay_ms = np.array([ev[s][0].elapsed_time(ev[s][1]) for s in sampled])
        dis_ms = np.array([ev[s][1].elapsed_time(ev[s][2]) for s in sampled])
        com_ms = np.array([ev[s][2].elapsed_time(ev[s][3]) for s in sampled])
    step_ms = wall * 1e3 / a.steps
    b = algorithmic_bytes(cfg)
    dc_bytes = b["dispatch"] + b["combine"]
    value = dc_bytes / (step_ms * 1e-3) / 1e9
    d_us, c_us, l_us = dis_ms.mean() * 1e3, com_ms.mean() * 1e3, lay_ms.mean() * 1e3
    if graph is not None:
        # a replayed graph has no per-kernel events: whole-step figures only
        # (lay_ms: each replay's time per step)
        dom, dom_bytes, dom_us = "layout+dispatch+combine (graph)", dc_bytes, l_us
        d_us = c_us = l_us = float("nan")
        traffic = None
    else:
        dom = "dispatch" if d_us >= c_us else "combine"
        dom_bytes, dom_us = (b["dispatch"], d_us) if dom == "dispatch" else (b["combine"], c_us)
        traffic = read_traffic(cfg["name"], dom)
    d_gbps = b["dispatch"] / (d_us * 1e-6) / 1e9
    c_gbps = b["combine"] / (c_us * 1e-6) / 1e9
    achieved = dom_bytes / (dom_us * 1e-6) / 1e9

    out = {
        "metric": "dispatch+combine effective GB/s (algorithmic bytes / whole-step time)",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8_e4m3+f32" if fp8 else "bf16",
        "data": "synthetic",
        "config": {"workload": cfg["name"], "T": T, "H": H, "E": E, "R": R, "k": k,
                   "payload": "fp8_e4m3" if fp8 else "bf16", "zipf_s": cfg["zipf_s"],
                   "force_frac": cfg["force_frac"], "parallelism": "1 GPU, R emulated ranks",
                   "layout": "packed" if capacity is None else f"fixed windows of {capacity}",
                   "graph": bool(graph is not None), "x_copies": n_x},
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBPS, 2),
        "tokens_per_s": round(T / (step_ms * 1e-3), 1),
        "layout_us": _num(l_us, 2),
        "dispatch_us": _num(d_us, 2),
        "combine_us": _num(c_us, 2),
        "phase_events": ({"every": every, "steps_timed": len(sampled)} if graph is None
                         else {"graph_steps": gsteps, "replays": len(replays)}),
        "dispatch_GBps": _num(d_gbps, 1),
        "combine_GBps": _num(c_gbps, 1),
        "dispatch_plus_combine_GBps": _num(dc_bytes / ((d_us + c_us) * 1e-6) / 1e9, 1),
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
        "cpu_baseline": None,
    }
    if graph is None and a.cold_reps > 0:
        # Cold caches: before each operation write a 1 GiB buffer, which
        # evicts the 256 MB MALL and the L2s, then time the operation alone.
        fl = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        evc = [[Event() for _ in range(6)]
               for _ in range(a.cold_reps)]
        for i, e in enumerate(evc):
            for j, op in enumerate((lambda: lay.run(idx_d), dispatch, combine)):
                fl.fill_((3 * i + j) & 0xFF)
                e[2 * j].record(stream)
                op()
                e[2 * j + 1].record(stream)
        torch.cuda.synchronize()
        del fl

        def pct(v):
            return {"median": round(float(np.median(v)), 2),
                    "p10": round(float(np.percentile(v, 10)), 2),
                    "p90": round(float(np.percentile(v, 90)), 2)}
        cl = np.array([e[0].elapsed_time(e[1]) for e in evc]) * 1e3
        cd = np.array([e[2].elapsed_time(e[3]) for e in evc]) * 1e3
        cc = np.array([e[4].elapsed_time(e[5]) for e in evc]) * 1e3
        dcm = float(np.median(cd)) + float(np.median(cc))
        out["cold"] = {"reps": a.cold_reps, "layout_us": pct(cl), "dispatch_us": pct(cd),
                       "combine_us": pct(cc),
                       "dispatch_plus_combine_GBps": round(dc_bytes / (dcm * 1e-6) / 1e9, 1)}
        out["warm_median_us"] = {"layout": round(float(np.median(lay_ms)) * 1e3, 2),
                                 "dispatch": round(float(np.median(dis_ms)) * 1e3, 2),
                                 "combine": round(float(np.median(com_ms)) * 1e3, 2)}
        if int(lay.status.item()) != 0:
            print("[bench] status word set in the cold pass", file=sys.stderr)
            return 1

    # Achievable-bandwidth reference on the same GPU: a plain device copy of
    # 1 GiB (read + write bytes / time), next to the 8 TB/s peak.
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = Event(), Event()
    e0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    out["hbm_copy_GBps"] = round(2 * src.numel() * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9, 1)
    del src, dst
    # ... and a copy that moves as many bytes as dispatch + combine
    half = max(16, dc_bytes // 2 // 16 * 16)
    src = torch.empty(half, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0.record(stream)
    for _ in range(10):
        dst.copy_(src)
    e1.record(stream)
    torch.cuda.synchronize()
    out["hbm_copy_equal_bytes_GBps"] = round(2 * half * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e9,
                                             1)
    del src, dst

    # Measured ceiling: what pure writes (dispatch's write bytes) and pure
    # reads (combine's read bytes) sustain on this GPU, and the rate each
    # kernel would reach with its reads and writes at those rates.
    legs = measure_stream_legs(dev, stream, b["combine_read"], b["dispatch_write"])
    ceil_d = stream_ceiling(b["dispatch_read"], b["dispatch_write"], legs["read_GBps"],
                            legs["write_GBps"])
    ceil_c = stream_ceiling(b["combine_read"], b["combine_write"], legs["read_GBps"],
                            legs["write_GBps"])
    out["ceiling"] = {
        "write_GBps": round(legs["write_GBps"], 1), "write_op": "torch fill_ (uint8)",
        "write_buffer_bytes": legs["write_buffer_bytes"],
        "read_GBps": round(legs["read_GBps"], 1), "read_op": legs["read_op"],
        "read_rates_GBps": legs["read_rates_GBps"], "read_buffer_bytes": legs["read_buffer_bytes"],
        "dispatch_GBps": round(ceil_d, 1), "combine_GBps": round(ceil_c, 1),
        "dispatch_frac": _num(d_gbps / ceil_d, 4), "combine_frac": _num(c_gbps / ceil_c, 4)}
    if graph is None:
        ach = ceil_d if dom == "dispatch" else ceil_c
        out["roofline"]["achievable"] = round(ach, 1)
        out["roofline"]["frac_of_achievable"] = round(achieved / ach, 4)

    if not a.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        cpu_s, reps = cpu_baseline(cfg, inp, capacity=capacity)
        out["cpu_baseline"] = {
            "value": round(dc_bytes / cpu_s / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"full workload ({'fixed-capacity ' if capacity else ''}layout+"
                      f"dispatch+combine), median of {reps} run(s), "
                      f"{cpu_s:.2f} s each, 1 thread, host CPU: {cpu_model()}",
            "tokens_per_s": round(T / cpu_s, 1), "host_nproc": os.cpu_count()}
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
