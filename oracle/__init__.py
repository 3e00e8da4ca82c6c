"""numpy front end of the CPU oracle (oracle/moe_oracle.cpp).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product package.  Every function
here marshals numpy arrays into the C oracle and back; all arithmetic is in the
C file, which cites the paper passage each function follows.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_DEFAULT_LIB = os.path.join(_HERE, "liboracle.so")
_LIB_PATH = _DEFAULT_LIB
_lib = None

P_ = ctypes.c_void_p
I32 = ctypes.c_int32
I64 = ctypes.c_int64


def use_library(path=None):
    """Load another build of the oracle (the mutation tests use this)."""
    global _lib, _LIB_PATH
    _lib = None
    _LIB_PATH = path or _DEFAULT_LIB


def lib():
    global _lib
    if _lib is None:
        if _LIB_PATH == _DEFAULT_LIB and not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(_LIB_PATH)
        L.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_to_double.restype = ctypes.c_double
        L.oracle_bf16_from_double.argtypes = [ctypes.c_double]
        L.oracle_bf16_from_double.restype = ctypes.c_uint16
        L.oracle_fp8e4m3_to_float.argtypes = [ctypes.c_uint8]
        L.oracle_fp8e4m3_to_float.restype = ctypes.c_float
        L.oracle_layout.argtypes = [P_, I64, I32, I32, I32, P_, P_, P_, P_, P_, P_, P_]
        L.oracle_plan.argtypes = [P_, I64, I32, I32, P_]
        L.oracle_layout_fixed.argtypes = [P_, I64, I32, I32, I32, I32, P_, P_, P_, P_, P_,
                                          P_, P_]
        L.oracle_dispatch.argtypes = [P_, I64, P_, I64, I64, I64, I32, I32, I32, P_, P_,
                                      P_, P_, P_, P_, P_]
        L.oracle_expert_scale.argtypes = [P_, P_, I64, I32, I32, I32, I32, I32, P_, P_,
                                          P_, P_]
        L.oracle_combine.argtypes = [P_, P_, I64, I32, I32, I32, I32, P_, P_, P_,
                                     P_, P_, P_]
        L.oracle_layout_dedup.argtypes = [P_, I64, I32, I32, I32, P_, P_, P_, P_, P_]
        L.oracle_expand.argtypes = [P_, P_, I64, I64, I64, I64, I32, I32, I32, P_, P_, P_,
                                    P_, P_, P_, P_, P_, P_, P_]
        L.oracle_combine_local.argtypes = [P_, P_, I64, I32, I32, I32, I32, P_, P_, P_, P_,
                                           P_, P_, P_, P_, P_]
        for f in ("oracle_layout", "oracle_layout_fixed", "oracle_plan", "oracle_dispatch",
                  "oracle_expert_scale", "oracle_combine", "oracle_layout_dedup",
                  "oracle_expand", "oracle_combine_local"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _ptr_table(arrays):
    tab = (ctypes.c_void_p * max(1, len(arrays)))()
    for i, a in enumerate(arrays):
        tab[i] = a.ctypes.data if a is not None else None
    return tab


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: bad arguments (rc={rc})")


# ---------------------------------------------------------------- formats
def bf16_to_double(bits) -> float:
    return lib().oracle_bf16_to_double(int(bits))


def bf16_from_double(v: float) -> int:
    return int(lib().oracle_bf16_from_double(float(v)))


def fp8e4m3_to_float(code: int) -> float:
    return float(lib().oracle_fp8e4m3_to_float(int(code)))


# ---------------------------------------------------------------- layout
def layout(topk_idx: np.ndarray, E: int, R: int) -> dict:
    """Token placement: counts, offsets, pos and row_src (int32 arrays)."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    out = dict(
        expert_count=np.zeros(E, np.int32), expert_offset=np.zeros(E + 1, np.int32),
        rank_count=np.zeros(R, np.int32), rank_offset=np.zeros(R + 1, np.int32),
        pos=np.zeros(T * k, np.int32), row_src=np.zeros(T * k, np.int32))
    st = np.zeros(1, np.uint32)
    rc = lib().oracle_layout(_p(idx), T, k, E, R, _p(out["expert_count"]),
                             _p(out["expert_offset"]), _p(out["rank_count"]),
                             _p(out["rank_offset"]), _p(out["pos"]),
                             _p(out["row_src"]), _p(st))
    _check(rc, "oracle_layout")
    out["status"] = int(st[0])
    return out


def layout_fixed(topk_idx: np.ndarray, E: int, R: int, C: int) -> dict:
    """Fixed-capacity placement: expert windows of C rows (row_src has E*C)."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    out = dict(
        expert_count=np.zeros(E, np.int32), expert_offset=np.zeros(E + 1, np.int32),
        rank_count=np.zeros(R, np.int32), rank_offset=np.zeros(R + 1, np.int32),
        pos=np.zeros(T * k, np.int32), row_src=np.zeros(max(1, E * C), np.int32))
    st = np.zeros(1, np.uint32)
    rc = lib().oracle_layout_fixed(_p(idx), T, k, E, R, C, _p(out["expert_count"]),
                                   _p(out["expert_offset"]), _p(out["rank_count"]),
                                   _p(out["rank_offset"]), _p(out["pos"]),
                                   _p(out["row_src"]), _p(st))
    _check(rc, "oracle_layout_fixed")
    out["row_src"] = out["row_src"][: E * C]
    out["status"] = int(st[0])
    return out


def plan(pos: np.ndarray, T: int, k: int, P: int) -> np.ndarray:
    """Byte-balanced part boundaries bound[P+1] over the token range."""
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    bound = np.zeros(P + 1, np.int32)
    _check(lib().oracle_plan(_p(pos), T, k, P, _p(bound)), "oracle_plan")
    return bound


# ---------------------------------------------------------------- dispatch
def dispatch(x_rows: np.ndarray, x_scale_rows, topk_idx, pos, rank_offset,
             E: int, R: int, recv_cap, sentinel: int = 0xA5, scale_pitch: int = 0):
    """Copy routed rows into R regions.

    x_rows: uint8 [T, row_bytes]; x_scale_rows: uint8 [T, scale_row_bytes] or
    None.  Regions are uint8 [recv_cap[r], row_bytes] pre-filled with
    `sentinel`; scale regions uint8 [recv_cap[r], scale_pitch] (0: packed).
    Returns (regions, scale_regions or None, status).
    """
    x_rows = np.ascontiguousarray(x_rows, dtype=np.uint8)
    T, rb = x_rows.shape
    k = topk_idx.shape[1]
    cap = np.ascontiguousarray(recv_cap, dtype=np.int32)
    regs = [np.full((int(c), rb), sentinel, np.uint8) for c in cap]
    sregs, srb, xs = None, 0, None
    if x_scale_rows is not None:
        xs = np.ascontiguousarray(x_scale_rows, dtype=np.uint8)
        srb = xs.shape[1]
        scale_pitch = scale_pitch or srb
        assert scale_pitch >= srb
        sregs = [np.full((int(c), scale_pitch), sentinel, np.uint8) for c in cap]
    st = np.zeros(1, np.uint32)
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    ro = np.ascontiguousarray(rank_offset, dtype=np.int32)
    rc = lib().oracle_dispatch(_p(x_rows), rb, _p(xs) if xs is not None else None,
                               srb, scale_pitch, T, k, E, R, _p(idx), _p(pos), _p(ro),
                               _ptr_table(regs),
                               _ptr_table(sregs) if sregs is not None else None,
                               _p(cap), _p(st))
    _check(rc, "oracle_dispatch")
    return regs, sregs, int(st[0])


# ---------------------------------------------------------------- expert
def expert_scale(regions, scale_regions, payload_fp8: bool, H: int, E: int,
                 R: int, identity: bool, expert_offset, rank_offset, recv_cap):
    """Stand-in expert: bf16 regions [recv_cap[r], H] of s_e * row.  Scale
    regions are [rows, scale_pitch] arrays (the pitch is their width)."""
    cap = np.ascontiguousarray(recv_cap, dtype=np.int32)
    outs = [np.zeros((int(c), H), np.uint16) for c in cap]
    eo = np.ascontiguousarray(expert_offset, dtype=np.int32)
    ro = np.ascontiguousarray(rank_offset, dtype=np.int32)
    pitch = scale_regions[0].shape[1] if scale_regions else 0
    rc = lib().oracle_expert_scale(
        _ptr_table(regions),
        _ptr_table(scale_regions) if scale_regions is not None else None, pitch,
        int(bool(payload_fp8)), H, E, R, int(bool(identity)), _p(eo), _p(ro),
        _p(cap), _ptr_table(outs))
    _check(rc, "oracle_expert_scale")
    return outs


# ---------------------------------------------------------------- combine
def combine(expert_y, topk_w, topk_idx, pos, rank_offset, recv_cap, E: int,
            R: int, H: int):
    """Top-k-weighted sum of expert outputs: (y uint16 [T,H], status)."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    w = np.ascontiguousarray(topk_w, dtype=np.float32)
    pos = np.ascontiguousarray(pos, dtype=np.int32)
    ro = np.ascontiguousarray(rank_offset, dtype=np.int32)
    cap = np.ascontiguousarray(recv_cap, dtype=np.int32)
    ys = [np.ascontiguousarray(a, dtype=np.uint16) for a in expert_y]
    y = np.zeros((T, H), np.uint16)
    st = np.zeros(1, np.uint32)
    rc = lib().oracle_combine(_ptr_table(ys), _p(w), T, H, k, E, R, _p(idx),
                              _p(pos), _p(ro), _p(cap), _p(y), _p(st))
    _check(rc, "oracle_combine")
    return y, int(st[0])



# ---------------------------------------------------------------- per-peer deduplication
def layout_dedup(topk_idx: np.ndarray, E: int, R: int) -> dict:
    """One row per (token, peer) pair: tok_count, tok_offset, tok_pos, tok_src."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    out = dict(tok_count=np.zeros(R, np.int32), tok_offset=np.zeros(R + 1, np.int32),
               tok_pos=np.zeros(T * k, np.int32), tok_src=np.zeros(T * k, np.int32))
    st = np.zeros(1, np.uint32)
    rc = lib().oracle_layout_dedup(_p(idx), T, k, E, R, _p(out["tok_count"]),
                                   _p(out["tok_offset"]), _p(out["tok_pos"]),
                                   _p(out["tok_src"]), _p(st))
    _check(rc, "oracle_layout_dedup")
    out["status"] = int(st[0])
    return out


def dispatch_dedup(x_rows, x_scale_rows, topk_idx, tok_pos, tok_offset, E: int, R: int,
                   dedup_cap, sentinel: int = 0xA5, scale_pitch: int = 0):
    """Send each (token, peer) pair once: the per-slot copy of dispatch()
    applied to the pair rows (tok_pos is -1 on all but a pair's first slot)."""
    return dispatch(x_rows, x_scale_rows, topk_idx, tok_pos, tok_offset, E, R, dedup_cap,
                    sentinel=sentinel, scale_pitch=scale_pitch)


def expand(dedup_regions, dedup_scale_regions, scale_row_bytes: int, topk_idx, pos,
           rank_offset, tok_pos, tok_offset, dedup_cap, E: int, R: int, recv_cap,
           sentinel: int = 0xA5):
    """Receiver-side permutation of pair rows into expert order.  Regions
    are uint8 [rows, row_bytes]; scale regions uint8 [rows, pitch], the pitch
    being their width.  Returns (regions, scale_regions or None, status)."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    dregs = [np.ascontiguousarray(a, dtype=np.uint8) for a in dedup_regions]
    rb = dregs[0].shape[1]
    cap = np.ascontiguousarray(recv_cap, dtype=np.int32)
    dcap = np.ascontiguousarray(dedup_cap, dtype=np.int32)
    regs = [np.full((int(c), rb), sentinel, np.uint8) for c in cap]
    dsregs, sregs, pitch = None, None, 0
    if dedup_scale_regions is not None:
        dsregs = [np.ascontiguousarray(a, dtype=np.uint8) for a in dedup_scale_regions]
        pitch = dsregs[0].shape[1]
        sregs = [np.full((int(c), pitch), sentinel, np.uint8) for c in cap]
    pos, ro, tp, to = (np.ascontiguousarray(a, dtype=np.int32)
                       for a in (pos, rank_offset, tok_pos, tok_offset))
    st = np.zeros(1, np.uint32)
    rc = lib().oracle_expand(_ptr_table(dregs),
                             _ptr_table(dsregs) if dsregs is not None else None,
                             rb, scale_row_bytes, pitch, T, k, E, R, _p(idx), _p(pos), _p(ro),
                             _p(tp), _p(to), _p(dcap), _ptr_table(regs),
                             _ptr_table(sregs) if sregs is not None else None, _p(cap),
                             _p(st))
    _check(rc, "oracle_expand")
    return regs, sregs, int(st[0])


def combine_local(expert_y, topk_w, topk_idx, pos, rank_offset, recv_cap, tok_pos,
                  tok_offset, part_cap, E: int, R: int, H: int, sentinel: int = 0xA5A5):
    """Per-(token, peer) partial sums: regions uint16 [part_cap[r], H]
    (rows no pair writes keep `sentinel`).  Returns (partials, status)."""
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    w = np.ascontiguousarray(topk_w, dtype=np.float32)
    pos, ro, cap, tp, to, pc = (np.ascontiguousarray(a, dtype=np.int32)
                                for a in (pos, rank_offset, recv_cap, tok_pos, tok_offset,
                                          part_cap))
    ys = [np.ascontiguousarray(a, dtype=np.uint16) for a in expert_y]
    parts = [np.full((int(c), H), sentinel, np.uint16) for c in pc]
    st = np.zeros(1, np.uint32)
    rc = lib().oracle_combine_local(_ptr_table(ys), _p(w), T, H, k, E, R, _p(idx), _p(pos),
                                    _p(ro), _p(cap), _p(tp), _p(to), _p(pc),
                                    _ptr_table(parts), _p(st))
    _check(rc, "oracle_combine_local")
    return parts, int(st[0])


def combine_dedup(partials, topk_idx, tok_pos, tok_offset, part_cap, E: int, R: int, H: int):
    """Source side of the deduplicated combine: the sum of a token's peer
    partials, i.e. combine() with unit weights over the pair rows."""
    T, k = np.asarray(topk_idx).shape
    return combine(partials, np.ones((T, k), np.float32), topk_idx, tok_pos, tok_offset,
                   part_cap, E, R, H)
