"""Pins that tie the CPU oracle to facts fixed outside the oracle.

Each pin checks one oracle function against something other than itself:
brute-force enumeration written from the definition, a library routine in a
special case (torch's float32->bf16 and float8_e4m3fn casts, numpy's stable
sort), a closed form, or an invariant of the operator.  The pins are plain
functions so that test_oracle_mutants.py can run all of them against oracle
builds with a planted mistake and show that every mistake fails at least one.

Paper passages: token placement, expert and peer windows -- Appendix D;
remote-slice transfers -- Section 6.1; byte-balanced partitioning --
Section 6.2 and Appendix B.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction

import numpy as np

import oracle
import workloads as wl

# ----------------------------------------------------------------- formats
# All finite bf16 values, non-negative half, in increasing order (bit patterns
# 0x0000..0x7F7F map monotonically to values).
_POS_BITS = np.arange(0, 0x7F80, dtype=np.uint32)
_POS_VALS = (_POS_BITS << 16).view(np.float32).astype(np.float64)


def _nearest_bf16_bruteforce(x: float) -> int:
    """Nearest bf16 to x by exact comparison, ties to the even pattern."""
    if math.isnan(x):
        return -1
    sign = 0x8000 if math.copysign(1.0, x) < 0 else 0
    ax = abs(x)
    bf_max = float(_POS_VALS[-1])                      # (2 - 2^-7) * 2^127
    overflow_at = Fraction(bf_max) + Fraction(2) ** 119  # half an ulp above
    if math.isinf(ax) or Fraction(ax) >= overflow_at:
        return sign | 0x7F80
    i = int(np.searchsorted(_POS_VALS, ax))
    cands = [c for c in (i - 1, i) if 0 <= c < len(_POS_VALS)]
    fx = Fraction(ax)
    best = min(cands, key=lambda c: (abs(Fraction(float(_POS_VALS[c])) - fx),
                                     int(_POS_BITS[c]) & 1))
    return sign | int(_POS_BITS[best])


def _format_probe_values():
    rng = np.random.Generator(np.random.PCG64(11))
    vals = [0.0, -0.0, 1.0, -1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8,
            1.0 + 2.0 ** -8 + 2.0 ** -30, 1.0 - 2.0 ** -10, 3.0e38, 3.4e38,
            float(_POS_VALS[-1]), float(_POS_VALS[-1]) * (1 + 2.0 ** -9),
            float(_POS_VALS[-1]) * (1 + 2.0 ** -9) * (1 - 2.0 ** -40),
            2.0 ** -126, 2.0 ** -133, 2.0 ** -134, 1.5 * 2.0 ** -134,
            2.0 ** -135, 3 * 2.0 ** -134, 2.0 ** -130 * 1.01, 1e-45, 5e-324,
            math.inf, -math.inf]
    # exact ties between consecutive bf16 values, both parities
    for b in (0x3F80, 0x3F81, 0x4000, 0x0001, 0x0080, 0x7F7E, 0x1234):
        lo, hi = float(_POS_VALS[b]), float(_POS_VALS[b + 1])
        vals += [(lo + hi) / 2, -(lo + hi) / 2]
    mant = rng.random(400) + 1.0
    expo = rng.integers(-140, 128, 400)
    sgn = rng.choice([-1.0, 1.0], 400)
    vals += list(sgn * np.ldexp(mant, expo))
    return vals


def pin_bf16_from_double_bruteforce():
    for v in _format_probe_values():
        got = oracle.bf16_from_double(v)
        want = _nearest_bf16_bruteforce(v)
        assert got == want, (v, hex(got), hex(want))
    assert oracle.bf16_from_double(math.nan) & 0x7FFF > 0x7F80


def pin_bf16_from_float_matches_torch():
    import torch
    rng = np.random.Generator(np.random.PCG64(12))
    f = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(5000) * 1e30).astype(np.float32),
        (rng.standard_normal(5000) * 1e-39).astype(np.float32),
        np.array([3.3895314e38, 3.4e38, 1e-45, -1e-45, 0.0], np.float32)])
    want = torch.from_numpy(f).to(torch.bfloat16).view(torch.int16).numpy()
    want = want.astype(np.uint16)
    got = np.array([oracle.bf16_from_double(float(v)) for v in f], np.uint16)
    assert np.array_equal(got, want)


def pin_bf16_to_double_exhaustive():
    bits = np.arange(0x10000, dtype=np.uint32)
    with np.errstate(invalid="ignore"):
        ref = (bits << 16).view(np.float32).astype(np.float64)
    got = np.array([oracle.bf16_to_double(int(b)) for b in bits])
    fin = np.isfinite(ref)
    assert np.array_equal(got[fin], ref[fin])
    assert np.array_equal(np.isnan(got), np.isnan(ref))


def pin_fp8_decode_matches_torch():
    import torch
    codes = np.arange(256, dtype=np.uint8)
    want = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy()
    got = np.array([oracle.fp8e4m3_to_float(int(c)) for c in codes], np.float32)
    assert np.array_equal(np.isnan(got), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.array_equal(got[ok], want[ok])
    # values fixed by the OCP E4M3FN definition
    assert oracle.fp8e4m3_to_float(0x7E) == 448.0
    assert oracle.fp8e4m3_to_float(0x01) == 2.0 ** -9
    assert oracle.fp8e4m3_to_float(0x38) == 1.0
    assert oracle.fp8e4m3_to_float(0xB8) == -1.0
    assert math.isnan(oracle.fp8e4m3_to_float(0x7F))


# ----------------------------------------------------------------- layout
def layout_bruteforce(idx: np.ndarray, E: int, R: int) -> dict:
    """Placement from its definition: a routed slot's row is the number of
    routed slots whose (expert, token, slot) key is lexicographically
    smaller.  Quadratic; small inputs only."""
    T, k = idx.shape
    L = E // R
    st = 0
    used = []
    for t in range(T):
        seen = set()
        for j in range(k):
            e = int(idx[t, j])
            if e == -1:
                continue
            if e < -1 or e >= E:
                st |= 1
                continue
            if e in seen:
                st |= 2
                continue
            seen.add(e)
            used.append((e, t, j))
    pos = -np.ones(T * k, np.int64)
    for (e, t, j) in used:
        pos[t * k + j] = sum(1 for key in used if key < (e, t, j))
    ec = np.array([sum(1 for u in used if u[0] == e) for e in range(E)])
    rcount = np.array([ec[r * L:(r + 1) * L].sum() for r in range(R)])
    eo = np.array([ec[:e].sum() for e in range(E + 1)])
    ro = np.array([eo[r * L] for r in range(R)] + [eo[E]])
    row_src = -np.ones(T * k, np.int64)
    for s in range(T * k):
        if pos[s] >= 0:
            row_src[pos[s]] = s
    return dict(expert_count=ec, expert_offset=eo, rank_count=rcount,
                rank_offset=ro, pos=pos, row_src=row_src, status=st)


def _assert_layout_equal(got, want, ctx):
    for key in ("expert_count", "expert_offset", "rank_count", "rank_offset",
                "pos", "row_src"):
        assert np.array_equal(np.asarray(got[key], np.int64),
                              np.asarray(want[key], np.int64)), (key, ctx)
    assert got["status"] == want["status"], ("status", ctx)


def pin_layout_exhaustive_tiny():
    """Every routing table with T*k <= 4 slots over values {-1..3} (E=4), plus
    a sweep including out-of-range values, for R in {1, 2, 4}."""
    E = 4
    for R in (1, 2, 4):
        for T, k in ((0, 1), (1, 1), (2, 1), (3, 1), (4, 1), (1, 2), (2, 2), (1, 4)):
            for vals in itertools.product(range(-1, E), repeat=T * k):
                idx = np.array(vals, np.int32).reshape(T, k)
                _assert_layout_equal(oracle.layout(idx, E, R),
                                     layout_bruteforce(idx, E, R), (R, vals))
        for vals in itertools.product((-2, -1, 0, 3, 4), repeat=4):
            idx = np.array(vals, np.int32).reshape(2, 2)
            _assert_layout_equal(oracle.layout(idx, E, R),
                                 layout_bruteforce(idx, E, R), (R, vals))


def pin_layout_random_bruteforce():
    rng = np.random.Generator(np.random.PCG64(21))
    for case in range(60):
        E = int(rng.choice([4, 8, 12, 16, 32]))
        R = int(rng.choice([r for r in (1, 2, 4, E) if E % r == 0]))
        k = int(rng.integers(1, min(E, 6) + 1))
        T = int(rng.integers(0, 24))
        idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) \
            if T else np.zeros((0, k), np.int32)
        if case % 3 == 0 and T:
            idx[rng.random(idx.shape) < 0.2] = -1
        if case % 7 == 0 and T:
            idx[0, 0] = E + 3
        if case % 5 == 0 and T and k > 1:
            idx[-1, 1] = idx[-1, 0]
        _assert_layout_equal(oracle.layout(idx, E, R), layout_bruteforce(idx, E, R),
                             case)


def pin_layout_equals_stable_sort():
    """Positions equal numpy's stable argsort of the routed slots by expert
    (slots flattened token-major): a library routine in the distinct-expert
    case."""
    rng = np.random.Generator(np.random.PCG64(22))
    for T, E, R, k in ((300, 64, 8, 6), (1000, 256, 64, 8), (257, 16, 4, 2)):
        idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
        idx[rng.random(idx.shape) < 0.1] = -1
        lay = oracle.layout(idx, E, R)
        flat = idx.ravel()
        used = np.nonzero(flat >= 0)[0]
        order = used[np.argsort(flat[used], kind="stable")]
        want_pos = -np.ones(T * k, np.int64)
        want_pos[order] = np.arange(len(order))
        assert np.array_equal(lay["pos"], want_pos)
        assert np.array_equal(lay["row_src"][:len(order)], order)
        assert np.all(lay["row_src"][len(order):] == -1)
        assert np.array_equal(lay["expert_count"], np.bincount(flat[used], minlength=E))


def check_layout_invariants(idx, E, R, lay):
    """Properties of any correct placement (used at full workload sizes)."""
    T, k = idx.shape
    L = E // R
    ec, eo = lay["expert_count"].astype(np.int64), lay["expert_offset"].astype(np.int64)
    rc, ro = lay["rank_count"].astype(np.int64), lay["rank_offset"].astype(np.int64)
    pos, row_src = lay["pos"].astype(np.int64), lay["row_src"].astype(np.int64)
    nvalid = int((idx >= 0).sum())
    assert ec.sum() == nvalid == rc.sum()
    assert eo[0] == 0 and eo[-1] == nvalid and np.all(np.diff(eo) == ec)
    assert np.array_equal(ro[:-1], eo[0:E:L]) and ro[-1] == nvalid
    assert np.array_equal(rc, ec.reshape(R, L).sum(1))
    used = pos >= 0
    assert np.array_equal(np.sort(pos[used]), np.arange(nvalid))
    assert np.array_equal(row_src[pos[used]], np.nonzero(used)[0])
    assert np.all(row_src[nvalid:] == -1)
    # rows of one expert window belong to that expert, in strictly increasing
    # token order
    e_of_row = idx.ravel()[row_src[:nvalid]]
    assert np.array_equal(e_of_row, np.repeat(np.arange(E), ec))
    tok = row_src[:nvalid] // k
    same = e_of_row[1:] == e_of_row[:-1]
    assert np.all(tok[1:][same] > tok[:-1][same])


def pin_layout_special_cases():
    rng = np.random.Generator(np.random.PCG64(23))
    T, E, k = 200, 16, 4
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    one = oracle.layout(idx, E, 1)          # R = 1: a single region
    assert np.array_equal(one["rank_offset"], [0, T * k])
    every = oracle.layout(idx, E, E)        # R = E: one expert per region
    assert np.array_equal(every["rank_count"], every["expert_count"])
    k1 = oracle.layout(idx[:, :1].copy(), E, 4)  # k = 1: a permutation of tokens
    assert np.array_equal(np.sort(k1["row_src"]), np.arange(T))
    empty = oracle.layout(np.zeros((0, k), np.int32), E, 4)
    assert empty["expert_offset"].sum() == 0 and empty["status"] == 0
    for R in (1, 4, E):
        check_layout_invariants(idx, E, R, oracle.layout(idx, E, R))


def pin_layout_slot_permutation_invariance():
    """Reordering the slots of a token moves its pos entries with them and
    changes nothing else."""
    rng = np.random.Generator(np.random.PCG64(24))
    T, E, R, k = 500, 32, 8, 5
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)
    perm = np.stack([rng.permutation(k) for _ in range(T)])
    idx2 = np.take_along_axis(idx, perm, axis=1)
    a, b = oracle.layout(idx, E, R), oracle.layout(idx2, E, R)
    for key in ("expert_count", "expert_offset", "rank_count", "rank_offset"):
        assert np.array_equal(a[key], b[key])
    assert np.array_equal(np.take_along_axis(a["pos"].reshape(T, k), perm, axis=1),
                          b["pos"].reshape(T, k))
    assert np.array_equal(a["row_src"] // k, b["row_src"] // k)


def layout_fixed_bruteforce(idx, E, R, C):
    """Fixed windows from the definition: a routed slot's rank within its
    expert is the number of earlier tokens routed to the same expert; it is
    placed at e*C + rank when rank < C."""
    T, k = idx.shape
    L = E // R
    base = layout_bruteforce(idx, E, R)     # validity and status bits 1, 2
    pos = -np.ones(T * k, np.int64)
    st = base["status"]
    count = np.zeros(E, np.int64)
    for t in range(T):
        for j in range(k):
            if base["pos"][t * k + j] < 0:
                continue
            e = int(idx[t, j])
            rank = sum(1 for tt in range(t) for jj in range(k)
                       if base["pos"][tt * k + jj] >= 0 and idx[tt, jj] == e)
            if rank < C:
                pos[t * k + j] = e * C + rank
                count[e] += 1
            else:
                st |= 4
    row_src = -np.ones(E * C, np.int64)
    for s_ in range(T * k):
        if pos[s_] >= 0:
            row_src[pos[s_]] = s_
    return dict(expert_count=count, expert_offset=np.arange(E + 1) * C,
                rank_count=count.reshape(R, L).sum(1), rank_offset=np.arange(R + 1) * L * C,
                pos=pos, row_src=row_src, status=st)


def pin_layout_fixed_bruteforce():
    rng = np.random.Generator(np.random.PCG64(25))
    for case in range(80):
        E = int(rng.choice([4, 8, 16]))
        R = int(rng.choice([r for r in (1, 2, 4) if E % r == 0]))
        k = int(rng.integers(1, min(E, 4) + 1))
        T = int(rng.integers(0, 20))
        C = int(rng.integers(0, 8))
        idx = np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32) \
            if T else np.zeros((0, k), np.int32)
        if case % 3 == 0 and T:
            idx[rng.random(idx.shape) < 0.2] = -1
        if case % 5 == 0 and T:
            idx[0, 0] = E + 1
        _assert_layout_equal(oracle.layout_fixed(idx, E, R, C),
                             layout_fixed_bruteforce(idx, E, R, C), case)


def pin_layout_fixed_large_capacity_equals_packed():
    """With C >= every expert's count, the fixed windows hold exactly the
    packed layout's rows, each window shifted to e*C."""
    idx, _ = wl.make_routing(wl.get("decode"))
    E, R = 256, 64
    packed = oracle.layout(idx, E, R)
    C = int(packed["expert_count"].max())
    fixed = oracle.layout_fixed(idx, E, R, C)
    assert fixed["status"] == 0
    assert np.array_equal(fixed["expert_count"], packed["expert_count"])
    e = np.where(idx.ravel() >= 0, idx.ravel(), 0)
    shift = e * C - packed["expert_offset"][e]
    assert np.array_equal(fixed["pos"], packed["pos"] + shift)


# ----------------------------------------------------------------- plan
def _plan_bruteforce(pos, T, k, P):
    cost = [1 + sum(1 for j in range(k) if pos[t * k + j] >= 0) for t in range(T)]
    a = [0]
    for c in cost:
        a.append(a[-1] + c)
    A = a[-1]
    return [min(t for t in range(T + 1) if a[t] * P >= p * A) for p in range(P + 1)]


def pin_plan_bruteforce_and_balance():
    rng = np.random.Generator(np.random.PCG64(31))
    for case in range(40):
        T = int(rng.integers(0, 40))
        k = int(rng.integers(1, 5))
        P = int(rng.integers(1, 50))
        pos = np.where(rng.random(T * k) < 0.3, -1, 0).astype(np.int32)
        got = oracle.plan(pos, T, k, P)
        assert list(got) == _plan_bruteforce(pos, T, k, P), case
    # balance at a full workload size: every token in exactly one part, each
    # part within one token of the ideal share
    idx, _ = wl.make_routing(wl.get("prefill"))
    T, k = idx.shape
    lay = oracle.layout(idx, 256, 64)
    for P in (1, 7, 4096, 20000):
        b = oracle.plan(lay["pos"], T, k, P).astype(np.int64)
        assert b[0] == 0 and b[-1] == T and np.all(np.diff(b) >= 0)
        cost = 1 + (lay["pos"].reshape(T, k) >= 0).sum(1)
        cp = np.concatenate([[0], np.cumsum(cost)])
        part = cp[b[1:]] - cp[b[:-1]]
        assert part.max() <= cp[-1] / P + cost.max()


def pin_plan_equal_units_match_lpt():
    """One memory tier and equal-size units: the list scheduler of Section
    6.2 puts ceil(U/C) units on the busiest core, and so does the plan."""
    for T, P in ((16384, 4096), (1000, 7), (5, 9), (4096, 4096)):
        k = 8
        pos = np.zeros(T * k, np.int32)
        b = oracle.plan(pos, T, k, P).astype(np.int64)
        # least-loaded-first assignment of T equal jobs to P cores
        loads = np.zeros(P, np.int64)
        for _ in range(min(T, 50000)):
            loads[np.argmin(loads)] += 1
        assert np.diff(b).max() == loads.max() == -(-T // P)


def _routed_slots(idx: np.ndarray, E: int) -> np.ndarray:
    """Routed slots per token, from the routing rules alone (an index in
    [0, E) that no earlier slot of the row repeats), not from the layout."""
    T, k = idx.shape
    n = np.zeros(T, np.int64)
    for t in range(T):
        seen = set()
        for e in idx[t]:
            if 0 <= e < E and e not in seen:
                n[t] += 1
            seen.add(int(e))
    return n


def pin_plan_mixed_costs_vs_list_scheduler():
    """Tokens of mixed cost (masked slots, whole rows masked, a block of
    rows with every slot masked): cut each token's payload into equal-cost
    units (one row read, one row per routed slot) and spread the units over
    P cores with the least-loaded list scheduler of Section 6.2 -- every
    core ends within one unit of A/P.  The plan keeps tokens whole, so each
    of its parts must carry A/P units to within one token's cost, with the
    costs counted from the routing rules, not from the layout under test."""
    E, R, k = 64, 16, 8
    rng = np.random.Generator(np.random.PCG64(77))
    for case, (T, P) in enumerate(((3000, 64), (777, 13), (4096, 512), (50, 7))):
        logits = rng.standard_normal((T, E)).astype(np.float32)
        idx = np.argsort(-logits, axis=1, kind="stable")[:, :k].astype(np.int32)
        idx[rng.random((T, k)) < 0.3] = -1       # scattered unused slots
        idx[: T // 3] = -1                       # a third of the batch unrouted
        idx[T // 2: T // 2 + 5, 1] = idx[T // 2: T // 2 + 5, 0]   # repeats
        cost = 1 + _routed_slots(idx, E)
        A = int(cost.sum())
        # least-loaded list scheduling of A equal units onto P cores
        loads = np.zeros(P, np.int64)
        for _ in range(A):
            loads[int(np.argmin(loads))] += 1
        assert loads.max() - loads.min() <= 1 and loads.sum() == A
        lay = oracle.layout(idx, E, R)
        b = oracle.plan(lay["pos"], T, k, P).astype(np.int64)
        assert b[0] == 0 and b[-1] == T and np.all(np.diff(b) >= 0), case
        cp = np.concatenate([[0], np.cumsum(cost)])
        part = cp[b[1:]] - cp[b[:-1]]
        slack = int(cost.max()) - 1
        assert part.max() <= loads.max() + slack, (case, part.max(), loads.max())
        assert part.min() >= loads.min() - slack, (case, part.min(), loads.min())
        assert part.sum() == A


# ----------------------------------------------------------------- dispatch
def _rows_u8(x):
    return np.ascontiguousarray(x).view(np.uint8).reshape(x.shape[0], -1)


def pin_dispatch_rows_are_source_rows():
    for cfg in (wl.custom(97, 40, 12, 3, 3, seed=3),
                wl.custom(64, 256, 16, 4, 2, payload=wl.FP8_E4M3, seed=4)):
        inp = wl.make_inputs(cfg)
        idx = wl.mask_slots(inp["topk_idx"], 0.15, seed=5)
        E, R, k = cfg["E"], cfg["R"], cfg["k"]
        lay = oracle.layout(idx, E, R)
        cap = lay["rank_count"] + 2             # spare rows keep the sentinel
        xr = _rows_u8(inp["x"])
        xs = _rows_u8(inp["x_scales"]) if inp["x_scales"] is not None else None
        regs, sregs, st = oracle.dispatch(xr, xs, idx, lay["pos"], lay["rank_offset"],
                                          E, R, cap)
        assert st == 0
        for r in range(R):
            n = int(lay["rank_count"][r])
            src = lay["row_src"][lay["rank_offset"][r]:lay["rank_offset"][r] + n] // k
            assert np.array_equal(regs[r][:n], xr[src])
            assert np.all(regs[r][n:] == 0xA5)
            if xs is not None:
                assert np.array_equal(sregs[r][:n], xs[src])
                assert np.all(sregs[r][n:] == 0xA5)


def pin_dispatch_pitched_scale_rows():
    """Scale rows spaced by a pitch: the scales, then zeros to the pitch; rows
    never written keep the sentinel."""
    cfg = wl.custom(80, 640, 16, 4, 3, payload=wl.FP8_E4M3, seed=8)
    inp = wl.make_inputs(cfg)
    lay = oracle.layout(inp["topk_idx"], 16, 4)
    cap = lay["rank_count"] + 1
    xs = _rows_u8(inp["x_scales"])
    sb = xs.shape[1]
    for pitch in (sb, 32, 128):
        _, sregs, st = oracle.dispatch(_rows_u8(inp["x"]), xs, inp["topk_idx"], lay["pos"],
                                       lay["rank_offset"], 16, 4, cap, scale_pitch=pitch)
        assert st == 0
        for r in range(4):
            n = int(lay["rank_count"][r])
            src = lay["row_src"][lay["rank_offset"][r]:lay["rank_offset"][r] + n] // 3
            assert sregs[r].shape == (int(cap[r]), pitch)
            assert np.array_equal(sregs[r][:n, :sb], xs[src])
            assert np.all(sregs[r][:n, sb:] == 0)
            assert np.all(sregs[r][n:] == 0xA5)


def pin_dispatch_capacity_overflow():
    cfg = wl.custom(50, 16, 8, 2, 2, seed=6)
    inp = wl.make_inputs(cfg)
    lay = oracle.layout(inp["topk_idx"], 8, 2)
    cap = lay["rank_count"].copy()
    cap[0] = max(0, cap[0] - 3)
    xr = _rows_u8(inp["x"])
    regs, _, st = oracle.dispatch(xr, None, inp["topk_idx"], lay["pos"],
                                  lay["rank_offset"], 8, 2, cap)
    assert st == 4
    src = lay["row_src"][:cap[0]] // 2
    assert np.array_equal(regs[0], xr[src])


# ----------------------------------------------------------------- combine
def _bf16_rows_to_f64(a):
    return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _torch_bf16_bits(f32):
    import torch
    return torch.from_numpy(np.ascontiguousarray(f32, np.float32)).to(
        torch.bfloat16).view(torch.int16).numpy().astype(np.uint16)


def _end_to_end(cfg, idx, w, identity, scale_pitch=0):
    inp = wl.make_inputs(cfg)
    E, R, H = cfg["E"], cfg["R"], cfg["H"]
    lay = oracle.layout(idx, E, R)
    cap = lay["rank_count"]
    fp8 = cfg["payload"] == wl.FP8_E4M3
    xs = _rows_u8(inp["x_scales"]) if fp8 else None
    regs, sregs, _ = oracle.dispatch(_rows_u8(inp["x"]), xs, idx, lay["pos"],
                                     lay["rank_offset"], E, R, cap, scale_pitch=scale_pitch)
    ey = oracle.expert_scale(regs, sregs, fp8, H, E, R, identity,
                             lay["expert_offset"], lay["rank_offset"], cap)
    y, st = oracle.combine(ey, w, idx, lay["pos"], lay["rank_offset"], cap, E, R, H)
    return inp, lay, ey, y, st


def pin_combine_identity_unit_weights_is_kx():
    """Identity expert, unit weights: y = bf16(k * x); for k a power of two
    this is x with its exponent raised, and torch's cast gives it for k=3."""
    for k in (2, 3, 8):
        cfg = wl.custom(70, 264, 16, 4, k, expert="identity", seed=7 + k)
        inp0 = wl.make_inputs(cfg)
        w = np.ones_like(inp0["topk_w"])
        inp, _, _, y, st = _end_to_end(cfg, inp0["topk_idx"], w, True)
        assert st == 0
        xf = (inp["x"].astype(np.uint32) << 16).view(np.float32)
        want = _torch_bf16_bits(xf * np.float32(k))
        want[want == 0x8000] = 0   # the sum starts from +0: -0 inputs give +0
        assert np.array_equal(y, want)


def pin_combine_identity_softmax_returns_x():
    """Identity expert with softmax weights (the tiny workload): the weights
    sum to 1 within float32 rounding, far below half a bf16 ulp, so y == x."""
    cfg = wl.get("tiny")
    inp0 = wl.make_inputs(cfg)
    inp, _, _, y, st = _end_to_end(cfg, inp0["topk_idx"], inp0["topk_w"], True)
    assert st == 0
    assert np.array_equal(y, inp["x"])


def pin_combine_scaled_closed_form():
    """Scaled experts: y ~= x * sum_j w_j (1 + 0.01 e_j) to within the two
    bf16 roundings (expert output and y), bf16 and fp8 payloads.  With all
    weights and scales positive the terms share x's sign, so the relative
    bound holds element-wise."""
    for cfg, pitch in ((wl.custom(300, 136, 32, 8, 4, seed=9), 0),
                       (wl.custom(100, 256, 16, 4, 3, payload=wl.FP8_E4M3, seed=10), 0),
                       (wl.custom(100, 256, 16, 4, 3, payload=wl.FP8_E4M3, seed=10), 128)):
        inp0 = wl.make_inputs(cfg)
        idx, w = inp0["topk_idx"], inp0["topk_w"]
        inp, _, _, y, st = _end_to_end(cfg, idx, w, False, scale_pitch=pitch)
        assert st == 0
        if cfg["payload"] == wl.BF16:
            xf = _bf16_rows_to_f64(inp["x"])
        else:
            import torch
            q = torch.from_numpy(inp["x"]).view(torch.float8_e4m3fn).double().numpy()
            xf = q * np.repeat(inp["x_scales"].astype(np.float64), 128, axis=1)
        s = 1.0 + 0.01 * idx.astype(np.float64)
        ref = xf * (w.astype(np.float64) * s).sum(1, keepdims=True)
        err = np.abs(_bf16_rows_to_f64(y) - ref)
        # two roundings to bf16 (8 significant bits, unit roundoff 2^-8): the
        # expert outputs and y; slack for the float32 steps
        assert np.all(err <= 1.01 * 2 * 2.0 ** -8 * np.abs(ref))


def pin_combine_weights_slots_and_masks():
    """Each slot contributes w_j * (its own expert row): checked slot by slot
    on random expert outputs, plus masked and capacity-dropped slots."""
    cfg = wl.custom(120, 64, 16, 4, 4, seed=12)
    inp = wl.make_inputs(cfg)
    E, R, H, k = 16, 4, 64, 4
    idx = wl.mask_slots(inp["topk_idx"], 0.2, seed=13)
    idx[5] = -1                                         # one token with no slot
    w = inp["topk_w"] * np.float32(3.0) - np.float32(1.0)  # signed weights
    lay = oracle.layout(idx, E, R)
    cap = lay["rank_count"].copy()
    cap[1] = max(0, cap[1] - 4)
    ey = [wl.random_bf16_rows(int(c), H, seed=20 + r) for r, c in enumerate(cap)]
    y, st = oracle.combine(ey, w, idx, lay["pos"], lay["rank_offset"], cap, E, R, H)
    assert st == 4
    assert np.all(y[5] == 0)
    ref = np.zeros((idx.shape[0], H))
    for t in range(idx.shape[0]):
        for j in range(k):
            p = lay["pos"][t * k + j]
            if p < 0:
                continue
            r = idx[t, j] // (E // R)
            loc = p - lay["rank_offset"][r]
            if loc < cap[r]:
                ref[t] += float(w[t, j]) * _bf16_rows_to_f64(ey[r][loc])
    assert np.array_equal(y, _bf16_bits_from_f64_bruteforce(ref))


def _bf16_bits_from_f64_bruteforce(a):
    """Round doubles to bf16 through an exact brute-force nearest search."""
    out = np.empty(a.shape, np.uint16)
    flat = a.ravel()
    o = out.ravel()
    for i, v in enumerate(flat):
        o[i] = _nearest_bf16_bruteforce(float(v))
    return out


def pin_combine_slot_permutation_invariance():
    cfg = wl.custom(200, 96, 16, 4, 4, seed=14)
    inp = wl.make_inputs(cfg)
    rng = np.random.Generator(np.random.PCG64(15))
    perm = np.stack([rng.permutation(4) for _ in range(200)])
    idx2 = np.take_along_axis(inp["topk_idx"], perm, axis=1)
    w2 = np.take_along_axis(inp["topk_w"], perm, axis=1)
    _, _, _, y1, _ = _end_to_end(cfg, inp["topk_idx"], inp["topk_w"], False)
    _, _, _, y2, _ = _end_to_end(cfg, idx2, w2, False)
    assert np.array_equal(y1, y2)


def pin_expert_scale_matches_torch():
    """The stand-in expert is one float32 multiply by s_e = 1 + 0.01 e (two
    for fp8: block scale first), rounded to bf16: torch's float32 arithmetic
    and cast give the same bits."""
    import torch
    for payload in (wl.BF16, wl.FP8_E4M3):
        cfg = wl.custom(90, 256, 16, 4, 2, payload=payload, seed=16)
        inp = wl.make_inputs(cfg)
        lay = oracle.layout(inp["topk_idx"], 16, 4)
        cap = lay["rank_count"]
        xs = _rows_u8(inp["x_scales"]) if payload else None
        regs, sregs, _ = oracle.dispatch(_rows_u8(inp["x"]), xs, inp["topk_idx"],
                                         lay["pos"], lay["rank_offset"], 16, 4, cap)
        ey = oracle.expert_scale(regs, sregs, bool(payload), 256, 16, 4, False,
                                 lay["expert_offset"], lay["rank_offset"], cap)
        for r in range(4):
            for i in range(int(cap[r])):
                g = lay["rank_offset"][r] + i
                e = int(inp["topk_idx"].ravel()[lay["row_src"][g]])
                se = torch.tensor(1.0, dtype=torch.float32) + \
                    torch.tensor(0.01, dtype=torch.float32) * float(e)
                if payload == wl.BF16:
                    v = torch.from_numpy(regs[r][i].view(np.uint16).copy()).view(
                        torch.bfloat16).float()
                else:
                    q = torch.from_numpy(regs[r][i].copy()).view(torch.float8_e4m3fn).float()
                    sc = torch.from_numpy(sregs[r][i].view(np.float32).copy())
                    v = q * sc.repeat_interleave(128)
                want = (v * se).to(torch.bfloat16).view(torch.int16).numpy()
                assert np.array_equal(ey[r][i], want.astype(np.uint16)), (payload, r, i)



# ------------------------------------------------------ per-peer deduplication
def layout_dedup_bruteforce(idx: np.ndarray, E: int, R: int) -> dict:
    """Deduplicated placement from its definition: the routed (token, peer)
    pairs, each pair's row = number of pairs with a smaller (peer, token)
    key, carried by the pair's first routed slot.  Quadratic; small inputs."""
    T, k = idx.shape
    L = E // R
    st = 0
    first_slot = {}                       # (r, t) -> first routed slot j
    for t in range(T):
        seen = set()
        for j in range(k):
            e = int(idx[t, j])
            if e == -1:
                continue
            if e < -1 or e >= E:
                st |= 1
                continue
            if e in seen:
                st |= 2
                continue
            seen.add(e)
            first_slot.setdefault((e // L, t), j)
    keys = list(first_slot)
    tok_pos = -np.ones(T * k, np.int64)
    tok_src = -np.ones(T * k, np.int64)
    for (r, t), j in first_slot.items():
        row = sum(1 for key in keys if key < (r, t))
        tok_pos[t * k + j] = row
        tok_src[row] = t * k + j
    cnt = np.array([sum(1 for key in keys if key[0] == r) for r in range(R)])
    off = np.concatenate([[0], np.cumsum(cnt)])
    return dict(tok_count=cnt, tok_offset=off, tok_pos=tok_pos, tok_src=tok_src, status=st)


def _assert_dedup_equal(got, want, ctx):
    for key in ("tok_count", "tok_offset", "tok_pos", "tok_src", "status"):
        assert np.array_equal(np.asarray(got[key], np.int64),
                              np.asarray(want[key], np.int64)), (key, ctx)


def pin_layout_dedup_exhaustive_tiny():
    """Every routing of 2 tokens x 2 slots over 4 experts on 2 peers, with
    unused (-1), out-of-range (-3, -2, 4) and repeated indices."""
    vals = [-3, -2, -1, 0, 1, 2, 3, 4]
    for combo in itertools.product(vals, repeat=4):
        idx = np.array(combo, np.int32).reshape(2, 2)
        got = oracle.layout_dedup(idx, 4, 2)
        _assert_dedup_equal(got, layout_dedup_bruteforce(idx, 4, 2), combo)


def pin_layout_dedup_random_bruteforce():
    """Random routings with masks, repeats and bad indices, several E/R."""
    rng = np.random.default_rng(31)
    for (T, k, E, R) in ((17, 3, 12, 3), (9, 5, 16, 4), (25, 4, 8, 8), (11, 6, 24, 2),
                         (13, 2, 6, 1)):
        idx = rng.integers(-3, E + 1, size=(T, k)).astype(np.int32)
        got = oracle.layout_dedup(idx, E, R)
        _assert_dedup_equal(got, layout_dedup_bruteforce(idx, E, R), (T, k, E, R))


def pin_layout_dedup_invariants_and_special_cases():
    """Peer counts are the numbers of distinct tokens per peer (numpy sets);
    with one expert per peer the deduplicated placement is the per-expert one;
    with k = 1 every slot is its own pair and the counts are the peer loads."""
    for cfg in (wl.custom(500, 64, 32, 8, 6, zipf_s=1.2, seed=41),
                wl.custom(300, 64, 16, 16, 4, seed=42),
                wl.custom(200, 64, 24, 6, 1, seed=43)):
        inp = wl.make_inputs(cfg)
        idx = wl.mask_slots(inp["topk_idx"], 0.1, seed=44)
        E, R, (T, k) = cfg["E"], cfg["R"], idx.shape
        L = E // R
        d = oracle.layout_dedup(idx, E, R)
        lay = oracle.layout(idx, E, R)
        for r in range(R):
            toks = np.unique(np.nonzero(((idx // L) == r) & (idx >= 0))[0])
            assert d["tok_count"][r] == len(toks)
            rows = d["tok_pos"][(d["tok_pos"] >= d["tok_offset"][r]) &
                                (d["tok_pos"] < d["tok_offset"][r + 1])]
            assert np.array_equal(np.sort(d["tok_src"][rows] // k), toks)
            # token order inside the peer window
            assert np.all(np.diff(d["tok_src"][d["tok_offset"][r]:d["tok_offset"][r + 1]]) > 0)
        assert np.all(d["tok_count"] <= lay["rank_count"])
        n = int(d["tok_offset"][-1])
        assert np.array_equal(np.sort(d["tok_pos"][d["tok_pos"] >= 0]), np.arange(n))
        if L == 1 or k == 1:
            assert np.array_equal(d["tok_count"], lay["rank_count"])
        if L == 1:
            assert np.array_equal(d["tok_pos"], lay["pos"])


def _dedup_chain(cfg, idx, w, identity, scale_pitch=0, dcap_delta=None):
    inp = wl.make_inputs(cfg)
    E, R, H = cfg["E"], cfg["R"], cfg["H"]
    fp8 = cfg["payload"] == wl.FP8_E4M3
    xs = _rows_u8(inp["x_scales"]) if fp8 else None
    lay = oracle.layout(idx, E, R)
    d = oracle.layout_dedup(idx, E, R)
    dcap = d["tok_count"].copy()
    if dcap_delta is not None:
        dcap = np.maximum(0, dcap + np.asarray(dcap_delta))
    dregs, dsregs, st_d = oracle.dispatch_dedup(_rows_u8(inp["x"]), xs, idx, d["tok_pos"],
                                                d["tok_offset"], E, R, dcap,
                                                scale_pitch=scale_pitch)
    cap = lay["rank_count"]
    srb = xs.shape[1] if fp8 else 0
    regs, sregs, st_e = oracle.expand(dregs, dsregs, srb, idx, lay["pos"], lay["rank_offset"],
                                      d["tok_pos"], d["tok_offset"], dcap, E, R, cap)
    out = dict(inp=inp, lay=lay, d=d, dcap=dcap, dregs=dregs, dsregs=dsregs, regs=regs,
               sregs=sregs, st_d=st_d, st_e=st_e)
    ey = oracle.expert_scale(regs, sregs, fp8, H, E, R, identity, lay["expert_offset"],
                             lay["rank_offset"], cap)
    parts, st_l = oracle.combine_local(ey, w, idx, lay["pos"], lay["rank_offset"], cap,
                                       d["tok_pos"], d["tok_offset"], d["tok_count"],
                                       E, R, H)
    y, st_y = oracle.combine_dedup(parts, idx, d["tok_pos"], d["tok_offset"],
                                   d["tok_count"], E, R, H)
    out.update(ey=ey, parts=parts, y=y, st_l=st_l, st_y=st_y)
    return out


def pin_dispatch_dedup_rows_and_expand_equals_dispatch():
    """Pair rows hold their token's row; expanding them into expert order
    gives byte for byte the per-slot dispatch (bf16, fp8 with packed and
    pitched scale rows, masked slots)."""
    for cfg, pitch in ((wl.custom(300, 72, 32, 8, 6, zipf_s=1.2, seed=51), 0),
                       (wl.custom(150, 256, 24, 6, 4, payload=wl.FP8_E4M3, seed=52), 0),
                       (wl.custom(150, 256, 24, 6, 4, payload=wl.FP8_E4M3, seed=53), 64)):
        inp0 = wl.make_inputs(cfg)
        idx = wl.mask_slots(inp0["topk_idx"], 0.15, seed=54)
        c = _dedup_chain(cfg, idx, inp0["topk_w"], True, scale_pitch=pitch)
        E, R = cfg["E"], cfg["R"]
        assert c["st_d"] == 0 and c["st_e"] == 0
        k = idx.shape[1]
        xr = _rows_u8(c["inp"]["x"])
        for r in range(R):
            a, b = c["d"]["tok_offset"][r], c["d"]["tok_offset"][r + 1]
            assert np.array_equal(c["dregs"][r], xr[c["d"]["tok_src"][a:b] // k])
        fp8 = cfg["payload"] == wl.FP8_E4M3
        xs = _rows_u8(c["inp"]["x_scales"]) if fp8 else None
        regs, sregs, st = oracle.dispatch(xr, xs, idx, c["lay"]["pos"], c["lay"]["rank_offset"],
                                          E, R, c["lay"]["rank_count"], scale_pitch=pitch)
        for r in range(R):
            assert np.array_equal(c["regs"][r], regs[r]), r
            if fp8:
                assert np.array_equal(c["sregs"][r], sregs[r]), r


def _pair_routing(T, k, E, R, seed):
    """Each token picks k/2 peers and both of two distinct experts on each."""
    rng = np.random.default_rng(seed)
    L = E // R
    idx = np.zeros((T, k), np.int32)
    for t in range(T):
        peers = rng.choice(R, size=k // 2, replace=False)
        col = []
        for r in peers:
            col.extend(r * L + rng.choice(L, size=2, replace=False))
        idx[t] = rng.permutation(np.array(col, np.int32))
    return idx


def pin_dedup_combine_pairs_identity_exact():
    """Identity experts, unit weights, experts in pairs per peer: each
    partial is 2x and y is k*x, both exact in bf16 (torch's casts)."""
    import torch
    for k in (2, 4, 8):
        cfg = wl.custom(60, 136, 32, 8, k, expert="identity", seed=60 + k)
        idx = _pair_routing(60, k, 32, 8, seed=61 + k)
        w = np.ones((60, k), np.float32)
        c = _dedup_chain(cfg, idx, w, True)
        assert c["st_l"] == 0 and c["st_y"] == 0
        xf = (c["inp"]["x"].astype(np.uint32) << 16).view(np.float32)
        want_y = _torch_bf16_bits(xf * np.float32(k))
        want_y[want_y == 0x8000] = 0
        assert np.array_equal(c["y"], want_y)
        want_p = _torch_bf16_bits(xf * np.float32(2))
        want_p[want_p == 0x8000] = 0
        for r in range(8):
            a, b = c["d"]["tok_offset"][r], c["d"]["tok_offset"][r + 1]
            assert np.array_equal(c["parts"][r], want_p[c["d"]["tok_src"][a:b] // k])


def pin_dedup_combine_unit_weights_matches_torch():
    """Identity experts, unit weights, any routing: partial_r = bf16(n_r x)
    with n_r the token's expert count on peer r, y = bf16(sum_r partial_r)
    (exact in float32 here), both cast by torch."""
    cfg = wl.custom(120, 72, 24, 6, 5, expert="identity", seed=71)
    inp0 = wl.make_inputs(cfg)
    idx = wl.mask_slots(inp0["topk_idx"], 0.1, seed=72)
    T, k = idx.shape
    c = _dedup_chain(cfg, idx, np.ones((T, k), np.float32), True)
    xf = (c["inp"]["x"].astype(np.uint32) << 16).view(np.float32)
    L = 4
    want_y = np.zeros((T, 72), np.float32)
    for t in range(T):
        ranks = [int(e) // L for e in idx[t] if e >= 0]
        for r in dict.fromkeys(ranks):
            pbits = _torch_bf16_bits(xf[t] * np.float32(ranks.count(r)))
            row = c["d"]["tok_pos"][t * k + [int(e) // L if e >= 0 else -1
                                             for e in idx[t]].index(r)]
            got = c["parts"][r][row - c["d"]["tok_offset"][r]]
            pb = pbits.copy()
            pb[pb == 0x8000] = 0
            assert np.array_equal(got, pb), (t, r)
            want_y[t] += (pbits.astype(np.uint32) << 16).view(np.float32)
    yb = _torch_bf16_bits(want_y)
    yb[yb == 0x8000] = 0
    assert np.array_equal(c["y"], yb)


def pin_dedup_combine_scaled_bound():
    """Scaled experts, softmax weights: partials within two bf16 roundings of
    x * sum over the peer's slots of w_j s_e, and y within three of
    x * sum_j w_j s_e (all terms share x's sign)."""
    cfg = wl.custom(200, 136, 32, 8, 6, zipf_s=1.2, seed=81)
    inp0 = wl.make_inputs(cfg)
    idx, w = inp0["topk_idx"], inp0["topk_w"]
    c = _dedup_chain(cfg, idx, w, False)
    xf = _bf16_rows_to_f64(c["inp"]["x"])
    s = (1.0 + 0.01 * idx.astype(np.float64)) * w.astype(np.float64)
    ref = xf * s.sum(1, keepdims=True)
    err = np.abs(_bf16_rows_to_f64(c["y"]) - ref)
    assert np.all(err <= 1.01 * 3 * 2.0 ** -8 * np.abs(ref))
    T, k = idx.shape
    L = 4
    for t in range(0, T, 7):
        for j0 in range(k):
            q = c["d"]["tok_pos"][t * k + j0]
            if q < 0:
                continue
            r = int(idx[t, j0]) // L
            sel = (idx[t] // L) == r
            pref = xf[t] * s[t, sel].sum()
            got = _bf16_rows_to_f64(c["parts"][r][q - c["d"]["tok_offset"][r]])
            assert np.all(np.abs(got - pref) <= 1.01 * 2 * 2.0 ** -8 * np.abs(pref))


def pin_dedup_capacity():
    """A short deduplicated region: rows past it are not written (sentinel
    kept), their slots are not expanded, and bit 4 is set on both sides."""
    cfg = wl.custom(100, 64, 16, 4, 3, seed=91)
    inp0 = wl.make_inputs(cfg)
    idx = inp0["topk_idx"]
    c = _dedup_chain(cfg, idx, inp0["topk_w"], True, dcap_delta=[0, -5, 0, 0])
    assert c["st_d"] == 4 and c["st_e"] == 4
    d, lay, k = c["d"], c["lay"], idx.shape[1]
    assert c["dregs"][1].shape[0] == d["tok_count"][1] - 5
    # slots whose pair row is past the short region keep the sentinel
    L = 4
    for s_ in range(idx.size):
        t, j = divmod(s_, k)
        if lay["pos"][s_] < 0 or int(idx[t, j]) // L != 1:
            continue
        q = [d["tok_pos"][t * k + jj] for jj in range(k)
             if d["tok_pos"][t * k + jj] >= 0 and int(idx[t, jj]) // L == 1][0]
        row = c["regs"][1][lay["pos"][s_] - lay["rank_offset"][1]]
        if q - d["tok_offset"][1] >= c["dcap"][1]:
            assert np.all(row == 0xA5)
        else:
            assert np.array_equal(row, _rows_u8(c["inp"]["x"])[t])


ALL_PINS = [v for k_, v in sorted(globals().items()) if k_.startswith("pin_")]
