"""Python binding of libep: the same calls as include/ep.h, marshalling only.

Every step of dispatch and combine runs in the library's HIP kernels or its DMA legs;
PyTorch provides device memory and streams.  Tensors must live on the current CUDA/HIP
device.  bf16 payload may be given as torch.bfloat16 or as raw 16-bit patterns
(torch.int16 / torch.uint16); only the bytes are used.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass
from typing import Optional

import numpy as np
import torch

from . import _lib
from ._lib import (EP_OK, EP_ERR_BAD_ROUTING, EP_ERR_TIMEOUT, EP_STAGING_HBM, EP_STAGING_PINNED_HOST,
                   EP_OUT_BF16, EP_OUT_F32, EP_SIM_ECHO, EP_SIM_FLAGS_ONLY)

MODE_PER_SENDER, MODE_DUPLEX, MODE_REMOTE_ONLY = _lib.EP_MODE_PER_SENDER, _lib.EP_MODE_DUPLEX, _lib.EP_MODE_REMOTE_ONLY
MODE_ACCUMULATE = _lib.EP_MODE_ACCUMULATE

__all__ = ["EPError", "Layout", "Staging", "SimPeers", "dispatch_layout", "layout_validate", "dispatch",
           "combine", "trace_enable", "trace_read", "trace_reset", "copy_probe", "stream_probe", "workspace_bytes",
           "pcie_probe", "MODE_PER_SENDER", "MODE_DUPLEX", "MODE_REMOTE_ONLY", "MODE_ACCUMULATE", "LocalLayout",
           "dispatch_layout_local", "pack", "combine_rows", "Dense", "allgather", "reducescatter",
           "round_advance", "round_read", "dispatch_graph", "combine_graph", "graph_legs_sdma"]

_PAYLOAD_DTYPES = (torch.bfloat16, torch.int16, torch.uint16)


class EPError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


_handle = None


def _lib_handle():
    global _handle
    if _handle is None:
        _handle = _lib.load()
    return _handle


def _check(status: int, what: str):
    if status != EP_OK:
        lib = _lib_handle()
        name = lib.ep_status_name(status).decode()
        raise EPError(status, f"{what}: {name}: {lib.ep_last_error().decode()}")


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)
_get_device = getattr(torch._C, "_cuda_getDevice", None) or torch.cuda.current_device


def _stream_ptr(stream=None) -> int:
    """Raw HIP stream handle: `stream` (torch stream or int handle), else the current stream."""
    if stream is None:
        if _raw_stream is not None:
            return _raw_stream(torch.cuda.current_device())
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _ptr(t: Optional[torch.Tensor]):
    return t.data_ptr() if t is not None and t.numel() else None


def _need(t: torch.Tensor, name: str, dtypes, ndim=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.device.index != _get_device():
        raise ValueError(f"{name} lives on {t.device}, not on the current device")
    if t.dtype not in dtypes:
        raise ValueError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")


def workspace_bytes(num_tokens: int, topk: int, num_experts: int) -> int:
    n = ctypes.c_size_t()
    _check(_lib_handle().ep_layout_workspace_bytes(num_tokens, topk, num_experts, ctypes.byref(n)),
           "ep_layout_workspace_bytes")
    return n.value


@dataclass
class Layout:
    num_tokens: int
    topk: int
    num_experts: int
    num_ranks: int
    expert_counts: torch.Tensor
    expert_offsets: torch.Tensor
    rank_counts: torch.Tensor
    rank_offsets: torch.Tensor
    slot_pos: torch.Tensor
    row_src: Optional[torch.Tensor]
    workspace: torch.Tensor


def _layout_buffers(T: int, k: int, num_experts: int, num_ranks: int, dev, with_row_src: bool,
                    out: Optional[Layout]) -> Layout:
    """The layout's output tensors and zero-filled workspace (reused when `out` fits)."""
    if out is not None and (out.num_tokens, out.topk, out.num_experts, out.num_ranks) == (T, k, num_experts,
                                                                                          num_ranks):
        return out
    i32 = dict(dtype=torch.int32, device=dev)
    return Layout(T, k, num_experts, num_ranks,
                  torch.empty(num_experts, **i32), torch.empty(num_experts + 1, **i32),
                  torch.empty(num_ranks, **i32), torch.empty(num_ranks + 1, **i32),
                  torch.empty(T * k, **i32), torch.empty(T * k, **i32) if with_row_src else None,
                  torch.zeros(workspace_bytes(T, k, num_experts) if 1 <= k <= num_experts
                              and 1 <= num_experts <= _lib.EP_MAX_EXPERTS else 256,
                              dtype=torch.uint8, device=dev))


def dispatch_layout(topk_idx: torch.Tensor, num_experts: int, num_ranks: int, *, with_row_src: bool = True,
                    out: Optional[Layout] = None, stream=None) -> Layout:
    """ep_dispatch_layout on a [T, k] int32 routing tensor; outputs are device tensors."""
    _need(topk_idx, "topk_idx", (torch.int32,), 2)
    T, k = topk_idx.shape
    out = _layout_buffers(T, k, num_experts, num_ranks, topk_idx.device, with_row_src, out)
    st = _lib_handle().ep_dispatch_layout(
        _ptr(topk_idx), T, k, num_experts, num_ranks, _ptr(out.expert_counts), _ptr(out.expert_offsets),
        _ptr(out.rank_counts), _ptr(out.rank_offsets), _ptr(out.slot_pos), _ptr(out.row_src),
        _ptr(out.workspace), out.workspace.numel(), _stream_ptr(stream))
    _check(st, "ep_dispatch_layout")
    return out


@dataclass
class LocalLayout:
    num_tokens: int
    topk: int
    num_experts: int
    e_lo: int
    e_hi: int
    local_counts: torch.Tensor
    local_offsets: torch.Tensor
    slot_pos: torch.Tensor
    row_src: Optional[torch.Tensor]
    workspace: torch.Tensor


def dispatch_layout_local(topk_idx: torch.Tensor, num_experts: int, e_lo: int, e_hi: int, *,
                          with_row_src: bool = True, out: Optional[LocalLayout] = None,
                          stream=None) -> LocalLayout:
    """ep_dispatch_layout_local: group N (gathered) tokens by the experts [e_lo, e_hi)."""
    _need(topk_idx, "topk_idx", (torch.int32,), 2)
    N, k = topk_idx.shape
    dev = topk_idx.device
    L = e_hi - e_lo
    if out is None or (out.num_tokens, out.topk, out.num_experts, out.e_lo, out.e_hi) != (N, k, num_experts, e_lo,
                                                                                          e_hi):
        i32 = dict(dtype=torch.int32, device=dev)
        # the window layout sorts all N*k entries over its L experts (k may exceed L: a token's
        # experts span several windows), so its workspace is that of N*k entries of top-1
        ws = workspace_bytes(N * k, 1, L) if N * k >= 1 and 1 <= L <= _lib.EP_MAX_EXPERTS else 256
        out = LocalLayout(N, k, num_experts, e_lo, e_hi, torch.empty(max(L, 1), **i32),
                          torch.empty(max(L, 0) + 1, **i32), torch.empty(N * k, **i32),
                          torch.empty(N * k, **i32) if with_row_src else None,
                          torch.zeros(max(ws, 256), dtype=torch.uint8, device=dev))
    _check(_lib_handle().ep_dispatch_layout_local(
        _ptr(topk_idx), N, k, num_experts, e_lo, e_hi, _ptr(out.local_counts), _ptr(out.local_offsets),
        _ptr(out.slot_pos), _ptr(out.row_src), _ptr(out.workspace), out.workspace.numel(), _stream_ptr(stream)),
        "ep_dispatch_layout_local")
    return out


def pack(x: torch.Tensor, slot_pos: torch.Tensor, out: torch.Tensor, *, topk: int, stream=None) -> torch.Tensor:
    """ep_pack: out[slot_pos[t*k+j]] = x[t] (slots outside [0, len(out)) skipped)."""
    _need(x, "x", _PAYLOAD_DTYPES, 2)
    _need(out, "out", _PAYLOAD_DTYPES, 2)
    _need(slot_pos, "slot_pos", (torch.int32,), 1)
    N, H = x.shape
    if out.shape[1] != H or slot_pos.numel() != N * topk:
        raise ValueError("shape mismatch between x, out and slot_pos")
    _check(_lib_handle().ep_pack(_ptr(x), N, H, topk, _ptr(slot_pos), _ptr(out), out.shape[0], _stream_ptr(stream)),
           "ep_pack")
    return out


def combine_rows(y: torch.Tensor, slot_pos: torch.Tensor, topk_w: torch.Tensor, out: torch.Tensor,
                 stream=None) -> torch.Tensor:
    """ep_combine_rows: out[t] = sum_j w[t, j] * y[slot_pos[t*k + j]] (fp32 accumulation)."""
    _need(topk_w, "topk_w", (torch.float32,), 2)
    _need(slot_pos, "slot_pos", (torch.int32,), 1)
    _need(out, "out", _PAYLOAD_DTYPES + (torch.float32,), 2)
    if y.numel():
        _need(y, "y", _PAYLOAD_DTYPES, 2)
    N, k = topk_w.shape
    H = out.shape[1]
    code = EP_OUT_F32 if out.dtype == torch.float32 else EP_OUT_BF16
    if y.numel() and y.shape[1] != H or slot_pos.numel() != N * k or out.shape[0] != N:
        raise ValueError("shape mismatch between y, out, topk_w and slot_pos")
    _check(_lib_handle().ep_combine_rows(_ptr(y), y.shape[0] if y.numel() else 0, _ptr(slot_pos), _ptr(topk_w), N, H,
                                         k, _ptr(out), code, _stream_ptr(stream)), "ep_combine_rows")
    return out


def layout_validate(layout: Layout, stream=None) -> None:
    """Synchronizes and raises EPError(EP_ERR_BAD_ROUTING) if the routing was rejected."""
    _check(_lib_handle().ep_layout_validate(_ptr(layout.workspace), _stream_ptr(stream)), "ep_layout_validate")


class Staging:
    """Library-owned send/recv buffers of one rank (ep_staging_alloc)."""

    def __init__(self, kind: str, max_rows: int, hidden: int, num_ranks: int, num_buffers: int = 2,
                 chunk_bytes: int = 0):
        kinds = {"hbm": EP_STAGING_HBM, "pinned": EP_STAGING_PINNED_HOST}
        if kind not in kinds:
            raise ValueError(f"kind must be one of {list(kinds)}")
        self.kind = kind
        handle = ctypes.c_void_p()
        _check(_lib_handle().ep_staging_alloc(kinds[kind], max_rows, hidden, num_ranks, num_buffers,
                                              chunk_bytes, ctypes.byref(handle)), "ep_staging_alloc")
        self.handle = handle
        self.views = [self._view(b) for b in range(num_buffers)]
        v = self.views[0]
        self.max_rows, self.hidden, self.num_ranks = v.max_rows, v.hidden, v.num_ranks
        self.num_buffers, self.row_bytes, self.chunk_bytes = v.num_buffers, v.row_bytes, v.chunk_bytes
        self.max_chunks = v.max_chunks

    def _view(self, buf: int) -> _lib.StagingView:
        v = _lib.StagingView()
        _check(_lib_handle().ep_staging_ptrs(self.handle, buf, ctypes.byref(v)), "ep_staging_ptrs")
        return v

    def close(self):
        if self.handle:
            _check(_lib_handle().ep_staging_free(self.handle), "ep_staging_free")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_mode(self, mode: int, self_rank: int = 0) -> None:
        """ep_staging_set_mode: EP_MODE_* bits (per-sender, duplex, remote-only)."""
        _check(_lib_handle().ep_staging_set_mode(self.handle, mode, self_rank), "ep_staging_set_mode")
        self.views = [self._view(b) for b in range(self.num_buffers)]

    def set_inbound(self, buf: int, rows_per_sender) -> None:
        """ep_staging_set_inbound: rows each other sender dispatches to this rank."""
        arr = (ctypes.c_int64 * self.num_ranks)(*[int(r) for r in rows_per_sender])
        _check(_lib_handle().ep_staging_set_inbound(self.handle, buf, arr), "ep_staging_set_inbound")

    # host views (pinned staging only): zero-copy numpy arrays over pinned memory
    _HOST_BUFFERS = {"send": "host_send", "recv": "host_recv", "in": "host_in", "ret": "host_ret"}
    _HOST_FLAGS = {"send_flags": "send_flags", "recv_flags": "recv_flags", "in_flags": "in_flags",
                   "ret_flags": "ret_flags", "in_landed": "in_landed", "recv_landed": "recv_landed",
                   "send_credits": "send_credits", "recv_credit": "recv_credit"}

    def host_array(self, which: str, buf: int = 0) -> np.ndarray:
        v = self.views[buf]
        if which in self._HOST_BUFFERS:
            ptr = getattr(v, self._HOST_BUFFERS[which])
            if not ptr:
                raise ValueError(f"host buffer {which!r} does not exist in this staging mode")
            return np.ctypeslib.as_array(ctypes.cast(ptr, ctypes.POINTER(ctypes.c_uint16)),
                                         shape=(self.max_rows, self.hidden))
        if which in self._HOST_FLAGS:
            ptr = getattr(v, self._HOST_FLAGS[which])
            if not ptr:
                raise ValueError("flags exist only with pinned staging")
            n = {"send_flags": self.max_chunks, "recv_credit": 1}.get(which, self.num_ranks)
            return np.ctypeslib.as_array(ctypes.cast(ptr, ctypes.POINTER(ctypes.c_uint32)), shape=(n,))
        if which == "in_offsets":
            return np.ctypeslib.as_array(ctypes.cast(v.in_offsets, ctypes.POINTER(ctypes.c_int64)),
                                         shape=(self.num_ranks + 1,))
        raise ValueError(which)

    def _dev_ptr(self, which: str, buf: int):
        v = self.views[buf]
        ptr = {"send": v.dev_send, "recv": v.dev_recv, "in": v.dev_in}.get(which)
        if not ptr:
            raise ValueError(f"device buffer {which!r} does not exist in this staging mode")
        return ptr

    def read_device(self, which: str, rows: int, buf: int = 0, stream=None) -> torch.Tensor:
        """Copy of the first `rows` rows of the device send, recv or in buffer (int16 bits)."""
        if not 0 <= rows <= self.max_rows:
            raise ValueError(f"rows must be in [0, {self.max_rows}]")
        ptr = self._dev_ptr(which, buf)
        out = torch.empty((rows, self.hidden), dtype=torch.int16, device="cuda")
        _check(_lib_handle().ep_memcpy(_ptr(out), ctypes.c_void_p(ptr), rows * self.row_bytes,
                                       _stream_ptr(stream)), "ep_memcpy")
        return out

    def write_device(self, which: str, rows: torch.Tensor, buf: int = 0, stream=None) -> None:
        """Copies a [rows, hidden] 16-bit device tensor into the device send, recv or in buffer."""
        _need(rows, "rows", _PAYLOAD_DTYPES, 2)
        if rows.shape[1] != self.hidden or rows.shape[0] > self.max_rows:
            raise ValueError("rows do not fit the staging buffer")
        ptr = self._dev_ptr(which, buf)
        _check(_lib_handle().ep_memcpy(ctypes.c_void_p(ptr), _ptr(rows), rows.numel() * 2, _stream_ptr(stream)),
               "ep_memcpy")

    def set_wait(self, timeout_us: int, sleep_units: int = 2) -> None:
        _check(_lib_handle().ep_staging_set_wait(self.handle, timeout_us, sleep_units), "ep_staging_set_wait")

    def status(self, stream=None) -> None:
        """Synchronizes; raises EPError(EP_ERR_TIMEOUT) if a flag wait expired."""
        _check(_lib_handle().ep_staging_status(self.handle, _stream_ptr(stream)), "ep_staging_status")


def _offsets_ptr(rank_offsets: Optional[torch.Tensor], staging: "Staging"):
    if rank_offsets is None:
        return None
    _need(rank_offsets, "rank_offsets", (torch.int32,), 1)
    if rank_offsets.numel() != staging.num_ranks + 1:
        raise ValueError("rank_offsets must hold num_ranks + 1 entries")
    return _ptr(rank_offsets)


def dispatch(x: torch.Tensor, slot_pos: torch.Tensor, staging: Staging, *, topk: int, buf: int = 0,
             epoch: int = 1, rank_offsets: Optional[torch.Tensor] = None, stream=None) -> None:
    """ep_dispatch: pack x [T, H] (bf16 bits) into staging buffer `buf` (and its host leg).
    rank_offsets (the layout's, int32 [R+1]) is required by the exchange modes."""
    _need(x, "x", _PAYLOAD_DTYPES, 2)
    _need(slot_pos, "slot_pos", (torch.int32,), 1)
    T, H = x.shape
    if slot_pos.numel() != T * topk:
        raise ValueError("slot_pos must hold T*topk entries")
    _check(_lib_handle().ep_dispatch(_ptr(x), T, H, topk, _ptr(slot_pos), _offsets_ptr(rank_offsets, staging),
                                     staging.handle, buf, epoch & 0xFFFFFFFF, _stream_ptr(stream)), "ep_dispatch")


def dispatch_fused(x: torch.Tensor, topk_idx: torch.Tensor, num_experts: int, num_ranks: int, staging: Staging, *,
                   buf: int = 0, epoch: int = 1, with_row_src: bool = True, out: Optional[Layout] = None,
                   stream=None) -> Layout:
    """ep_dispatch_fused: dispatch_layout then dispatch in one call (one kernel for few
    experts); returns the layout, as dispatch_layout does."""
    _need(topk_idx, "topk_idx", (torch.int32,), 2)
    _need(x, "x", _PAYLOAD_DTYPES, 2)
    T, k = topk_idx.shape
    if x.shape[0] != T:
        raise ValueError("x and topk_idx must have the same number of tokens")
    out = _layout_buffers(T, k, num_experts, num_ranks, topk_idx.device, with_row_src, out)
    _check(_lib_handle().ep_dispatch_fused(
        _ptr(topk_idx), T, k, num_experts, num_ranks, _ptr(out.expert_counts), _ptr(out.expert_offsets),
        _ptr(out.rank_counts), _ptr(out.rank_offsets), _ptr(out.slot_pos), _ptr(out.row_src),
        _ptr(out.workspace), out.workspace.numel(), _ptr(x), x.shape[1], staging.handle, buf, epoch & 0xFFFFFFFF,
        _stream_ptr(stream)), "ep_dispatch_fused")
    return out


def combine(staging: Staging, slot_pos: torch.Tensor, topk_w: torch.Tensor, *, out: Optional[torch.Tensor] = None,
            out_dtype: torch.dtype = torch.bfloat16, buf: int = 0, epoch: int = 1,
            rank_offsets: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """ep_combine: out [T, H] = sum_j w[t, j] * recv[slot_pos[t*k + j]] (fp32 accumulate)."""
    _need(topk_w, "topk_w", (torch.float32,), 2)
    _need(slot_pos, "slot_pos", (torch.int32,), 1)
    T, k = topk_w.shape
    H = staging.hidden
    if out is None:
        out = torch.empty((T, H), dtype=out_dtype, device=topk_w.device)
    if out.dtype == torch.float32:
        code = EP_OUT_F32
    elif out.dtype in _PAYLOAD_DTYPES:
        code = EP_OUT_BF16
    else:
        raise ValueError("out must be bf16 (or 16-bit bits) or float32")
    _need(out, "out", (out.dtype,), 2)
    if tuple(out.shape) != (T, H) or slot_pos.numel() != T * k:
        raise ValueError("shape mismatch between out, topk_w and slot_pos")
    _check(_lib_handle().ep_combine(staging.handle, buf, epoch & 0xFFFFFFFF, _ptr(slot_pos),
                                    _offsets_ptr(rank_offsets, staging), _ptr(topk_w), T, H, k,
                                    _ptr(out), code, _stream_ptr(stream)), "ep_combine")
    return out


class Dense:
    """Dense collectives of one rank (ep_dense_alloc): All-Gather / Reduce-Scatter staging."""

    def __init__(self, max_tokens: int, hidden: int, num_ranks: int, self_rank: int = 0, num_buffers: int = 2,
                 block_dtype: torch.dtype = torch.bfloat16):
        handle = ctypes.c_void_p()
        code = EP_OUT_F32 if block_dtype == torch.float32 else EP_OUT_BF16
        _check(_lib_handle().ep_dense_alloc(max_tokens, hidden, num_ranks, self_rank, num_buffers, code,
                                            ctypes.byref(handle)), "ep_dense_alloc")
        self.handle = handle
        self.views = []
        for b in range(num_buffers):
            v = _lib.DenseView()
            _check(_lib_handle().ep_dense_get(handle, b, ctypes.byref(v)), "ep_dense_get")
            self.views.append(v)
        self.max_tokens, self.hidden, self.num_ranks, self.self_rank = max_tokens, hidden, num_ranks, self_rank
        self.num_buffers = num_buffers
        self.block_dtype = torch.float32 if code == EP_OUT_F32 else torch.bfloat16

    def close(self):
        if self.handle:
            _check(_lib_handle().ep_dense_free(self.handle), "ep_dense_free")
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def set_policy(self, per_sender: bool = False, timeout_us: int = 10_000_000, host_threads: int = 0) -> None:
        _check(_lib_handle().ep_dense_set_policy(self.handle, MODE_PER_SENDER if per_sender else 0, timeout_us,
                                                 host_threads), "ep_dense_set_policy")

    def status(self, stream=None) -> None:
        _check(_lib_handle().ep_dense_status(self.handle, _stream_ptr(stream)), "ep_dense_status")

    def bytes_moved(self):
        up, down = ctypes.c_int64(), ctypes.c_int64()
        _check(_lib_handle().ep_dense_bytes(self.handle, ctypes.byref(up), ctypes.byref(down)), "ep_dense_bytes")
        return up.value, down.value

    _HOST = {"ag": ("host_ag", False), "rs_out": ("host_rs_out", True), "rs_in": ("host_rs_in", True)}
    _FLAGS = ("ag_flags", "ag_landed", "rs_out_flags", "rs_in_flags", "rs_landed")

    def host_array(self, which: str, buf: int = 0) -> np.ndarray:
        """[R * max_tokens, H] view of a pinned host buffer (uint16 bits, or float32 blocks)."""
        v = self.views[buf]
        if which in self._FLAGS:
            return np.ctypeslib.as_array(ctypes.cast(getattr(v, which), ctypes.POINTER(ctypes.c_uint32)),
                                         shape=(self.num_ranks,))
        field, is_block = self._HOST[which]
        ctype = ctypes.c_float if is_block and self.block_dtype == torch.float32 else ctypes.c_uint16
        return np.ctypeslib.as_array(ctypes.cast(getattr(v, field), ctypes.POINTER(ctype)),
                                     shape=(self.num_ranks * self.max_tokens, self.hidden))

    def device_rows(self, which: str, rows: int, buf: int = 0, stream=None) -> torch.Tensor:
        """Copy of the first `rows` rows of dev_gathered ("gathered") or dev_rs_in ("rs_in")."""
        if not 0 <= rows <= self.num_ranks * self.max_tokens:
            raise ValueError(f"rows must be in [0, {self.num_ranks * self.max_tokens}]")
        v = self.views[buf]
        if which == "gathered":
            ptr, dt, rb = v.dev_gathered, torch.int16, v.row_bytes
        else:
            ptr, dt, rb = v.dev_rs_in, (torch.float32 if self.block_dtype == torch.float32 else torch.int16), \
                v.block_row_bytes
        out = torch.empty((rows, self.hidden), dtype=dt, device="cuda")
        _check(_lib_handle().ep_memcpy(_ptr(out), ctypes.c_void_p(ptr), rows * rb, _stream_ptr(stream)), "ep_memcpy")
        return out


def allgather(dense: Dense, x: torch.Tensor, *, buf: int = 0, epoch: int = 1, stream=None) -> None:
    """ep_allgather: this rank's shard x [T, H] -> gathered rows of every rank."""
    _need(x, "x", _PAYLOAD_DTYPES, 2)
    T, H = x.shape
    if H != dense.hidden:
        raise ValueError("hidden size differs from the staging's")
    _check(_lib_handle().ep_allgather(dense.handle, buf, epoch & 0xFFFFFFFF, _ptr(x), T, _stream_ptr(stream)),
           "ep_allgather")


def reducescatter(dense: Dense, blocks: torch.Tensor, *, num_tokens: int, out: Optional[torch.Tensor] = None,
                  out_dtype: torch.dtype = torch.bfloat16, reduce_on_host: bool = False, buf: int = 0,
                  epoch: int = 1, stream=None) -> torch.Tensor:
    """ep_reducescatter: blocks [R*T, H] (block dtype) -> out [T, H], the sum for this rank's shard."""
    T, H = num_tokens, dense.hidden
    block_dtypes = (torch.float32,) if dense.block_dtype == torch.float32 else _PAYLOAD_DTYPES
    _need(blocks, "blocks", block_dtypes, 2)
    if tuple(blocks.shape) != (dense.num_ranks * T, H):
        raise ValueError("blocks must be [R*T, H]")
    if out is None:
        out = torch.empty((T, H), dtype=out_dtype, device=blocks.device)
    _need(out, "out", _PAYLOAD_DTYPES + (torch.float32,), 2)
    if tuple(out.shape) != (T, H):
        raise ValueError("out must be [T, H]")
    code = EP_OUT_F32 if out.dtype == torch.float32 else EP_OUT_BF16
    _check(_lib_handle().ep_reducescatter(dense.handle, buf, epoch & 0xFFFFFFFF, _ptr(blocks), T,
                                          1 if reduce_on_host else 0, _ptr(out), code, _stream_ptr(stream)),
           "ep_reducescatter")
    return out


def round_advance(staging: Staging, stream=None) -> None:
    """ep_round_advance: next graph-replayed round (device-side counter)."""
    _check(_lib_handle().ep_round_advance(staging.handle, _stream_ptr(stream)), "ep_round_advance")


def round_read(staging: Staging) -> int:
    r = ctypes.c_uint32()
    _check(_lib_handle().ep_round_read(staging.handle, ctypes.byref(r)), "ep_round_read")
    return r.value


def graph_legs_sdma(staging: Staging, on: bool = True) -> None:
    """ep_graph_legs_sdma: the host legs of graph-replayed rounds on SDMA engines (a library
    thread) instead of the compute units; call before capturing the rounds."""
    _check(_lib_handle().ep_graph_legs_sdma(staging.handle, 1 if on else 0), "ep_graph_legs_sdma")


def dispatch_graph(x: torch.Tensor, slot_pos: torch.Tensor, staging: Staging, *, topk: int, stream=None) -> None:
    """ep_dispatch_graph: pack x into the pinned send buffer of set round % 2 (replay-safe)."""
    _need(x, "x", _PAYLOAD_DTYPES, 2)
    _need(slot_pos, "slot_pos", (torch.int32,), 1)
    T, H = x.shape
    if slot_pos.numel() != T * topk:
        raise ValueError("slot_pos must hold T*topk entries")
    _check(_lib_handle().ep_dispatch_graph(_ptr(x), T, H, topk, _ptr(slot_pos), staging.handle, _stream_ptr(stream)),
           "ep_dispatch_graph")


def combine_graph(staging: Staging, slot_pos: torch.Tensor, topk_w: torch.Tensor, out: torch.Tensor,
                  stream=None) -> torch.Tensor:
    """ep_combine_graph: reduce the returned rows of set round % 2 straight from pinned memory."""
    _need(topk_w, "topk_w", (torch.float32,), 2)
    _need(slot_pos, "slot_pos", (torch.int32,), 1)
    _need(out, "out", _PAYLOAD_DTYPES + (torch.float32,), 2)
    T, k = topk_w.shape
    code = EP_OUT_F32 if out.dtype == torch.float32 else EP_OUT_BF16
    if tuple(out.shape) != (T, staging.hidden) or slot_pos.numel() != T * k:
        raise ValueError("shape mismatch between out, topk_w and slot_pos")
    _check(_lib_handle().ep_combine_graph(staging.handle, _ptr(slot_pos), _ptr(topk_w), T, staging.hidden, k,
                                          _ptr(out), code, _stream_ptr(stream)), "ep_combine_graph")
    return out


class SimPeers:
    """Host thread standing in for the peer ranks of a pinned staging (include/ep_sim.h)."""

    def __init__(self, staging, echo: bool = False, graph_rows: Optional[int] = None, graph_delay_us: int = 0):
        handle = ctypes.c_void_p()
        if graph_rows is not None:
            _check(_lib_handle().ep_sim_graph_start(staging.handle, graph_rows, graph_delay_us, 1 if echo else 0,
                                                    ctypes.byref(handle)), "ep_sim_graph_start")
        elif isinstance(staging, Dense):
            _check(_lib_handle().ep_sim_dense_start(staging.handle, ctypes.byref(handle)), "ep_sim_dense_start")
        else:
            _check(_lib_handle().ep_sim_peers_start(staging.handle, EP_SIM_ECHO if echo else EP_SIM_FLAGS_ONLY,
                                                    ctypes.byref(handle)), "ep_sim_peers_start")
        self.handle = handle
        self.staging = staging  # keep the staging alive while the thread reads it

    def wait_round(self, round_: int, timeout_ms: int = 60000) -> None:
        """Graph rounds: block until the peers finished round `round_`."""
        _check(_lib_handle().ep_sim_graph_wait(self.handle, round_ & 0xFFFFFFFF, timeout_ms), "ep_sim_graph_wait")

    def post_dense(self, buf: int, epoch: int, phase: str) -> None:
        """Dense staging: announce the other ranks' shards ("ag") or blocks ("rs")."""
        _check(_lib_handle().ep_sim_dense_post(self.handle, buf, epoch & 0xFFFFFFFF, 0 if phase == "ag" else 1),
               "ep_sim_dense_post")

    def post(self, buf: int, epoch: int, rows: int, delay_us: int = 0) -> None:
        _check(_lib_handle().ep_sim_peers_post(self.handle, buf, epoch & 0xFFFFFFFF, rows, delay_us),
               "ep_sim_peers_post")

    def set_delays(self, inbound_us=None, return_us=None) -> None:
        """Per-sender delays (microseconds) for rounds posted from now on."""
        R = self.staging.num_ranks

        def arr(v):
            return None if v is None else (ctypes.c_int64 * R)(*[int(t) for t in v])
        _check(_lib_handle().ep_sim_peers_set_delays(self.handle, arr(inbound_us), arr(return_us)),
               "ep_sim_peers_set_delays")

    def drain(self, timeout_ms: int = 60000) -> None:
        _check(_lib_handle().ep_sim_peers_drain(self.handle, timeout_ms), "ep_sim_peers_drain")

    def close(self) -> None:
        if self.handle:
            _lib_handle().ep_sim_peers_stop(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def trace_enable(on: bool = True) -> None:
    _check(_lib_handle().ep_trace_enable(1 if on else 0), "ep_trace_enable")


def trace_reset() -> None:
    _check(_lib_handle().ep_trace_reset(), "ep_trace_reset")


def trace_read() -> dict:
    """{name: {count, total_ms, mean_ms, min_ms, max_ms, p10_ms, p50_ms, p90_ms}} of the traced
    launches so far."""
    cap = 64
    arr = (_lib.TraceStat * cap)()
    n = ctypes.c_int32()
    _check(_lib_handle().ep_trace_read(arr, cap, ctypes.byref(n)), "ep_trace_read")
    out = {}
    for i in range(n.value):
        s = arr[i]
        out[s.name.decode()] = dict(count=s.count, total_ms=s.total_ms, mean_ms=s.total_ms / max(1, s.count),
                                    min_ms=s.min_ms, max_ms=s.max_ms, p10_ms=s.p10_ms, p50_ms=s.p50_ms,
                                    p90_ms=s.p90_ms)
    return out


def copy_probe(dst: torch.Tensor, src: torch.Tensor, stream=None) -> None:
    for t, name in ((dst, "dst"), (src, "src")):
        _need(t, name, (t.dtype,))
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst smaller than src")
    _check(_lib_handle().ep_copy_probe(_ptr(dst), _ptr(src), nbytes, _stream_ptr(stream)), "ep_copy_probe")


def stream_probe(dst: torch.Tensor, src: Optional[torch.Tensor], units: int, row_bytes: int, reads: int, writes: int,
                 store_policy: int = 0, stream=None) -> None:
    """ep_stream_probe: `units` units each reading `reads` rows and writing `writes` rows of
    row_bytes (sequential addresses), on device tensors large enough for them; store_policy
    0 non-temporal, 1 device-scope write-through, 2 write-through with the non-temporal hint."""
    need_src, need_dst = units * reads * row_bytes, units * writes * row_bytes if writes else 1024
    if dst.nbytes < need_dst or (reads and (src is None or src.nbytes < need_src)):
        raise ValueError("stream_probe: buffers too small for the units asked for")
    _check(_lib_handle().ep_stream_probe(_ptr(dst), _ptr(src) if reads else None, units, row_bytes, reads, writes,
                                         int(store_policy), _stream_ptr(stream)), "ep_stream_probe")


def pcie_probe(host: torch.Tensor, dev: torch.Tensor, nbytes: int, dirs: int) -> float:
    """ep_pcie_probe: GB/s over PCIe on the exchange's SDMA engines (dirs: 1 = device->host,
    2 = host->device, 3 = both at once).  host (pinned) and dev hold 2*nbytes each."""
    if host.is_cuda or not host.is_pinned() or not host.is_contiguous():
        raise ValueError("host must be a contiguous pinned host tensor")
    _need(dev, "dev", (dev.dtype,))
    if host.numel() * host.element_size() < 2 * nbytes or dev.numel() * dev.element_size() < 2 * nbytes:
        raise ValueError("host and dev must hold 2*nbytes")
    g = ctypes.c_double()
    _check(_lib_handle().ep_pcie_probe(_ptr(host), _ptr(dev), nbytes, dirs, ctypes.byref(g)), "ep_pcie_probe")
    return g.value
