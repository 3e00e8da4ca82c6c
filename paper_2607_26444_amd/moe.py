"""ctypes binding of libmoe (include/moe.h).

Argument marshalling only: every function passes device pointers of torch
tensors and the current HIP stream to the C entry point of the same name;
all work runs in the library's kernels.  torch is imported before the
library is loaded so that both use the one HIP runtime already in the
process.  There is no fallback: without libmoe.so every call raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmoe.so")

MOE_OK = 0
MOE_EINVAL = -1
MOE_EALIGN = -2
MOE_EWORKSPACE = -3
MOE_ELAUNCH = -4

MOE_DTYPE_BF16 = 0
MOE_DTYPE_FP8_E4M3 = 1

MOE_STATUS_BAD_INDEX = 1
MOE_STATUS_DUP_INDEX = 2
MOE_STATUS_CAPACITY = 4
MOE_STATUS_LAYOUT_SYNC = 8

MOE_MAX_K = 32
MOE_MAX_EXPERTS = 1024
MOE_FP8_BLOCK = 128
MOE_PLAN_PARTS = 12288

MOE_POLICY_BALANCED = 0
MOE_POLICY_ROWS = 1
MOE_POLICY_BY_RANK = 2
MOE_POLICY_DYNAMIC = 3
MOE_POLICY_STATIC = 4

# Entry points declared in include/moe.h.
EXPORTS = ("moe_version", "moe_strerror", "moe_last_hip_error", "moe_wall_clock_khz",
           "moe_layout_workspace_bytes", "moe_layout", "moe_layout_fixed", "moe_dispatch",
           "moe_dispatch_ex", "moe_combine", "moe_combine_ex", "moe_expert_scale",
           "moe_layout_dedup_workspace_bytes", "moe_layout_dedup", "moe_dispatch_dedup",
           "moe_expand", "moe_combine_local", "moe_combine_dedup", "moe_layout_scratch")

_lib = None
P = ctypes.c_void_p
I32 = ctypes.c_int
I64 = ctypes.c_int64
SZ = ctypes.c_size_t


class MoeError(RuntimeError):
    def __init__(self, fn, code):
        msg = lib().moe_strerror(code).decode()
        if code == MOE_ELAUNCH:
            msg += f" (hipError {lib().moe_last_hip_error()})"
        super().__init__(f"{fn}: {msg} [{code}]")
        self.code = code


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2607_26444_amd.build` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        L.moe_version.restype = I32
        L.moe_strerror.argtypes = [I32]
        L.moe_strerror.restype = ctypes.c_char_p
        L.moe_last_hip_error.restype = I32
        L.moe_wall_clock_khz.argtypes = [ctypes.POINTER(I32)]
        L.moe_wall_clock_khz.restype = I32
        L.moe_layout_workspace_bytes.argtypes = [I64, I32, I32, I32, ctypes.POINTER(SZ)]
        L.moe_layout.argtypes = [P, I64, I32, I32, I32, P, P, P, P, P, P, P, SZ, P, P]
        L.moe_layout_fixed.argtypes = [P, I64, I32, I32, I32, I32, P, P, P, P, P, P, P, SZ, P,
                                       P]
        L.moe_dispatch.argtypes = [P, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P, I32,
                                   P, P, SZ, P, P]
        L.moe_combine.argtypes = [P, P, I64, I32, I32, I32, I32, P, P, P, P, P, P, SZ, P, P]
        L.moe_dispatch_ex.argtypes = [P, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P, P,
                                      I32, P, P, SZ, P, I32, I32, P, I32, P]
        L.moe_combine_ex.argtypes = [P, P, I64, I32, I32, I32, I32, P, P, P, P, P, P, SZ, P,
                                     I32, I32, P, I32, P]
        L.moe_expert_scale.argtypes = [P, P, I32, I32, I32, I32, I32, I32, P, P, P, P, I64, P]
        L.moe_layout_dedup_workspace_bytes.argtypes = [I64, I32, I32, I32, ctypes.POINTER(SZ)]
        L.moe_layout_dedup.argtypes = [P, I64, I32, I32, I32, P, P, P, P, P, SZ, P, P]
        L.moe_dispatch_dedup.argtypes = [P, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P,
                                         I32, P, P, SZ, P, P]
        L.moe_expand.argtypes = [P, P, I32, I64, I32, I32, I32, I32, P, P, P, P, P, P, P, P,
                                 I32, P, P, SZ, P, P]
        L.moe_combine_local.argtypes = [P, P, I64, I32, I32, I32, I32, P, P, P, P, P, P, P, P,
                                        P, SZ, P, P]
        L.moe_combine_dedup.argtypes = [P, I64, I32, I32, I32, I32, P, P, P, P, P, P, SZ, P, P]
        L.moe_layout_scratch.argtypes = [P, I64, I32, I32, I32, P, P, P, P, P, P, P,
                                         ctypes.POINTER(P), ctypes.POINTER(SZ), P]
        for f in ("moe_layout_scratch", "moe_layout_workspace_bytes", "moe_layout", "moe_layout_fixed", "moe_dispatch",
                  "moe_dispatch_ex", "moe_combine", "moe_combine_ex", "moe_expert_scale",
                  "moe_layout_dedup_workspace_bytes", "moe_layout_dedup", "moe_dispatch_dedup",
                  "moe_expand", "moe_combine_local", "moe_combine_dedup"):
            getattr(L, f).restype = I32
        _lib = L
    return _lib


def _ptr(t):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("libmoe takes device tensors only")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _check(fn, rc):
    if rc != MOE_OK:
        raise MoeError(fn, rc)


def moe_version() -> int:
    return lib().moe_version()


def moe_wall_clock_khz() -> int:
    out = I32(0)
    _check("moe_wall_clock_khz", lib().moe_wall_clock_khz(ctypes.byref(out)))
    return out.value


def moe_layout_workspace_bytes(T: int, k: int, E: int, R: int) -> int:
    out = SZ(0)
    _check("moe_layout_workspace_bytes",
           lib().moe_layout_workspace_bytes(T, k, E, R, ctypes.byref(out)))
    return out.value


def moe_layout(topk_idx, E, R, expert_count, expert_offset, rank_count, rank_offset,
               pos, row_src, workspace, status, stream=None):
    T, k = topk_idx.shape
    _check("moe_layout", lib().moe_layout(
        _ptr(topk_idx), T, k, E, R, _ptr(expert_count), _ptr(expert_offset),
        _ptr(rank_count), _ptr(rank_offset), _ptr(pos), _ptr(row_src), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), _stream(stream)))


class DeviceBuffer:
    """A device address and size the library owns (the workspace that
    moe_layout_scratch returns), passed where the bindings take a tensor."""

    is_cuda = True

    def __init__(self, ptr: int, nbytes: int):
        self.ptr, self.nbytes = int(ptr), int(nbytes)

    def data_ptr(self) -> int:
        return self.ptr

    def numel(self) -> int:
        return self.nbytes

    def element_size(self) -> int:
        return 1


def moe_layout_scratch(topk_idx, E, R, expert_count, expert_offset, rank_count, rank_offset,
                       pos, row_src, status, stream=None) -> DeviceBuffer:
    """moe_layout into the library's own workspace; returns that workspace
    for this batch's dispatch and combine."""
    T, k = topk_idx.shape
    ws, nbytes = P(), SZ(0)
    _check("moe_layout_scratch", lib().moe_layout_scratch(
        _ptr(topk_idx), T, k, E, R, _ptr(expert_count), _ptr(expert_offset),
        _ptr(rank_count), _ptr(rank_offset), _ptr(pos), _ptr(row_src), _ptr(status),
        ctypes.byref(ws), ctypes.byref(nbytes), _stream(stream)))
    return DeviceBuffer(ws.value, nbytes.value)


def moe_layout_fixed(topk_idx, E, R, capacity, expert_count, expert_offset, rank_count,
                     rank_offset, pos, row_src, workspace, status, stream=None):
    T, k = topk_idx.shape
    _check("moe_layout_fixed", lib().moe_layout_fixed(
        _ptr(topk_idx), T, k, E, R, capacity, _ptr(expert_count), _ptr(expert_offset),
        _ptr(rank_count), _ptr(rank_offset), _ptr(pos), _ptr(row_src), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), _stream(stream)))


def moe_dispatch(x, x_scales, dtype, H, E, R, topk_idx, pos, rank_offset, recv_x,
                 recv_scales, recv_cap, workspace, status, stream=None, scale_pitch=0):
    T, k = topk_idx.shape
    _check("moe_dispatch", lib().moe_dispatch(
        _ptr(x), _ptr(x_scales), dtype, T, H, k, E, R, _ptr(topk_idx), _ptr(pos),
        _ptr(rank_offset), _ptr(recv_x), _ptr(recv_scales), scale_pitch, _ptr(recv_cap),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(status),
        _stream(stream)))


def moe_dispatch_ex(x, x_scales, dtype, H, E, R, topk_idx, pos, rank_offset, row_src,
                    recv_x, recv_scales, recv_cap, workspace, status, policy=MOE_POLICY_BALANCED,
                    trace=None, stream=None, scale_pitch=0, waves=0):
    T, k = topk_idx.shape
    _check("moe_dispatch_ex", lib().moe_dispatch_ex(
        _ptr(x), _ptr(x_scales), dtype, T, H, k, E, R, _ptr(topk_idx), _ptr(pos),
        _ptr(rank_offset), _ptr(row_src), _ptr(recv_x), _ptr(recv_scales), scale_pitch,
        _ptr(recv_cap), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(status), policy, waves, _ptr(trace), 0 if trace is None else trace.numel() // 2,
        _stream(stream)))


def moe_combine_ex(expert_y, topk_w, H, E, R, topk_idx, pos, rank_offset, recv_cap, y,
                   workspace, status, policy=MOE_POLICY_BALANCED, trace=None, stream=None,
                   waves=0):
    T, k = topk_idx.shape
    _check("moe_combine_ex", lib().moe_combine_ex(
        _ptr(expert_y), _ptr(topk_w), T, H, k, E, R, _ptr(topk_idx), _ptr(pos),
        _ptr(rank_offset), _ptr(recv_cap), _ptr(y), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), policy, waves,
        _ptr(trace), 0 if trace is None else trace.numel() // 2, _stream(stream)))


def moe_combine(expert_y, topk_w, H, E, R, topk_idx, pos, rank_offset, recv_cap, y,
                workspace, status, stream=None):
    T, k = topk_idx.shape
    _check("moe_combine", lib().moe_combine(
        _ptr(expert_y), _ptr(topk_w), T, H, k, E, R, _ptr(topk_idx), _ptr(pos),
        _ptr(rank_offset), _ptr(recv_cap), _ptr(y), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), _stream(stream)))


def moe_expert_scale(recv_x, recv_scales, dtype, H, E, R, identity, expert_offset,
                     rank_offset, recv_cap, out_y, max_rows, stream=None, scale_pitch=0):
    _check("moe_expert_scale", lib().moe_expert_scale(
        _ptr(recv_x), _ptr(recv_scales), scale_pitch, dtype, H, E, R, int(bool(identity)),
        _ptr(expert_offset), _ptr(rank_offset), _ptr(recv_cap), _ptr(out_y), max_rows,
        _stream(stream)))


# ------------------------------------------------ per-peer deduplicated path
def moe_layout_dedup_workspace_bytes(T: int, k: int, E: int, R: int) -> int:
    out = SZ(0)
    _check("moe_layout_dedup_workspace_bytes",
           lib().moe_layout_dedup_workspace_bytes(T, k, E, R, ctypes.byref(out)))
    return out.value


def moe_layout_dedup(topk_idx, E, R, tok_count, tok_offset, tok_pos, tok_src, workspace,
                     status, stream=None):
    T, k = topk_idx.shape
    _check("moe_layout_dedup", lib().moe_layout_dedup(
        _ptr(topk_idx), T, k, E, R, _ptr(tok_count), _ptr(tok_offset), _ptr(tok_pos),
        _ptr(tok_src), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(status), _stream(stream)))


def moe_dispatch_dedup(x, x_scales, dtype, H, E, R, topk_idx, tok_pos, tok_offset, recv_x,
                       recv_scales, recv_cap, workspace, status, stream=None, scale_pitch=0):
    T, k = topk_idx.shape
    _check("moe_dispatch_dedup", lib().moe_dispatch_dedup(
        _ptr(x), _ptr(x_scales), dtype, T, H, k, E, R, _ptr(topk_idx), _ptr(tok_pos),
        _ptr(tok_offset), _ptr(recv_x), _ptr(recv_scales), scale_pitch, _ptr(recv_cap),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(status),
        _stream(stream)))


def moe_expand(dedup_x, dedup_scales, dtype, H, E, R, topk_idx, pos, rank_offset, tok_pos,
               tok_offset, dedup_cap, recv_x, recv_scales, recv_cap, workspace, status,
               stream=None, scale_pitch=0):
    T, k = topk_idx.shape
    _check("moe_expand", lib().moe_expand(
        _ptr(dedup_x), _ptr(dedup_scales), dtype, T, H, k, E, R, _ptr(topk_idx), _ptr(pos),
        _ptr(rank_offset), _ptr(tok_pos), _ptr(tok_offset), _ptr(dedup_cap), _ptr(recv_x),
        _ptr(recv_scales), scale_pitch, _ptr(recv_cap), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _ptr(status), _stream(stream)))


def moe_combine_local(expert_y, topk_w, H, E, R, topk_idx, pos, rank_offset, recv_cap,
                      tok_pos, tok_offset, part_cap, partial, workspace, status, stream=None):
    T, k = topk_idx.shape
    _check("moe_combine_local", lib().moe_combine_local(
        _ptr(expert_y), _ptr(topk_w), T, H, k, E, R, _ptr(topk_idx), _ptr(pos),
        _ptr(rank_offset), _ptr(recv_cap), _ptr(tok_pos), _ptr(tok_offset), _ptr(part_cap),
        _ptr(partial), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(status), _stream(stream)))


def moe_combine_dedup(partial, H, E, R, topk_idx, tok_pos, tok_offset, part_cap, y, workspace,
                      status, stream=None):
    T, k = topk_idx.shape
    _check("moe_combine_dedup", lib().moe_combine_dedup(
        _ptr(partial), T, H, k, E, R, _ptr(topk_idx), _ptr(tok_pos), _ptr(tok_offset),
        _ptr(part_cap), _ptr(y), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _ptr(status), _stream(stream)))


# ------------------------------------------------------------ buffer plumbing
class Layout:
    """Device outputs of moe_layout (capacity None) or moe_layout_fixed
    (windows of `capacity` rows per expert) for one batch shape."""

    def __init__(self, T, k, E, R, device="cuda", capacity=None):
        i32 = dict(dtype=torch.int32, device=device)
        self.T, self.k, self.E, self.R, self.capacity = T, k, E, R, capacity
        self.expert_count = torch.empty(E, **i32)
        self.expert_offset = torch.empty(E + 1, **i32)
        self.rank_count = torch.empty(R, **i32)
        self.rank_offset = torch.empty(R + 1, **i32)
        self.pos = torch.empty(max(1, T * k), **i32)
        rows = T * k if capacity is None else E * capacity
        self.row_src = torch.empty(max(1, rows), **i32)
        nbytes = moe_layout_workspace_bytes(T, k, E, R)
        # torch's caching allocator returns 512-byte aligned blocks
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        assert self.workspace.data_ptr() % 256 == 0
        self.status = torch.zeros(1, dtype=torch.int32, device=device)

    def run(self, topk_idx, stream=None):
        if self.capacity is None:
            moe_layout(topk_idx, self.E, self.R, self.expert_count, self.expert_offset,
                       self.rank_count, self.rank_offset, self.pos, self.row_src,
                       self.workspace, self.status, stream)
        else:
            moe_layout_fixed(topk_idx, self.E, self.R, self.capacity, self.expert_count,
                             self.expert_offset, self.rank_count, self.rank_offset, self.pos,
                             self.row_src, self.workspace, self.status, stream)

    def plan(self):
        """The partition plan bound[MOE_PLAN_PARTS + 1] (a view of the workspace)."""
        return self.workspace[: (MOE_PLAN_PARTS + 1) * 4].view(torch.int32)


class DedupLayout:
    """Device outputs of moe_layout_dedup for one batch shape."""

    def __init__(self, T, k, E, R, device="cuda"):
        i32 = dict(dtype=torch.int32, device=device)
        self.T, self.k, self.E, self.R = T, k, E, R
        self.tok_count = torch.empty(R, **i32)
        self.tok_offset = torch.empty(R + 1, **i32)
        self.tok_pos = torch.empty(max(1, T * k), **i32)
        self.tok_src = torch.empty(max(1, T * k), **i32)
        nbytes = moe_layout_dedup_workspace_bytes(T, k, E, R)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        assert self.workspace.data_ptr() % 256 == 0
        self.status = torch.zeros(1, dtype=torch.int32, device=device)

    def run(self, topk_idx, stream=None):
        moe_layout_dedup(topk_idx, self.E, self.R, self.tok_count, self.tok_offset,
                         self.tok_pos, self.tok_src, self.workspace, self.status, stream)

    def plan(self):
        return self.workspace[: (MOE_PLAN_PARTS + 1) * 4].view(torch.int32)


class Regions:
    """R receive regions carved from one allocation, each 4 KiB aligned, with
    a device table of their base addresses (the emulated ranks)."""

    ALIGN = 4096

    def __init__(self, rows, row_bytes, device="cuda", guard_bytes=0, fill=None):
        self.rows = [int(r) for r in rows]
        self.row_bytes = int(row_bytes)
        self.guard = int(guard_bytes)
        offs, cur = [], self.guard
        for n in self.rows:
            cur = (cur + self.ALIGN - 1) // self.ALIGN * self.ALIGN
            offs.append(cur)
            cur += n * self.row_bytes + self.guard
        total = (cur + self.ALIGN - 1) // self.ALIGN * self.ALIGN + self.ALIGN
        self.buf = torch.empty(total, dtype=torch.uint8, device=device)
        if fill is not None:
            self.buf.fill_(fill)
        base = self.buf.data_ptr()
        pad = (-base) % self.ALIGN
        self.offsets = [o + pad for o in offs]
        self.table = torch.tensor([base + o for o in self.offsets], dtype=torch.int64,
                                  device=device)
        self.cap = torch.tensor(self.rows, dtype=torch.int32, device=device)

    def region(self, r):
        o = self.offsets[r]
        return self.buf[o: o + self.rows[r] * self.row_bytes].view(
            self.rows[r], self.row_bytes)
