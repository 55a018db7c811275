"""ctypes declarations of libep.so (include/ep.h and include/ep_sim.h).

Loading fails loudly when the library has not been built: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libep.so")

EP_OK, EP_ERR_INVALID_ARG, EP_ERR_BAD_ROUTING, EP_ERR_HIP, EP_ERR_OOM, EP_ERR_TIMEOUT = range(6)
EP_STAGING_HBM, EP_STAGING_PINNED_HOST = 0, 1
EP_OUT_BF16, EP_OUT_F32 = 0, 1
EP_SIM_FLAGS_ONLY, EP_SIM_ECHO = 0, 1
EP_MODE_PER_SENDER, EP_MODE_DUPLEX, EP_MODE_REMOTE_ONLY, EP_MODE_ACCUMULATE = 1, 2, 4, 8
ABI_VERSION = 6
EP_MAX_EXPERTS = 2048

c_i32, c_i64, c_u32, c_size, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t, ctypes.c_void_p
c_i32p = ctypes.POINTER(ctypes.c_int32)


class StagingView(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("num_ranks", c_i32), ("num_buffers", c_i32), ("hidden", c_i32),
                ("max_rows", c_i64), ("row_bytes", c_i64), ("buffer_bytes", c_i64), ("chunk_bytes", c_i64),
                ("max_chunks", c_i32),
                ("dev_send", c_vp), ("dev_recv", c_vp), ("host_send", c_vp), ("host_recv", c_vp),
                ("send_flags", c_vp), ("recv_flags", c_vp),
                ("mode", c_u32), ("self_rank", c_i32), ("dev_in", c_vp), ("host_in", c_vp), ("host_ret", c_vp),
                ("in_flags", c_vp), ("ret_flags", c_vp), ("in_landed", c_vp), ("recv_landed", c_vp),
                ("in_offsets", c_vp), ("send_credits", c_vp), ("recv_credit", c_vp)]


class DenseView(ctypes.Structure):
    _fields_ = [("num_ranks", c_i32), ("self_rank", c_i32), ("num_buffers", c_i32), ("hidden", c_i32),
                ("block_dtype", c_i32), ("max_tokens", c_i64), ("row_bytes", c_i64), ("block_row_bytes", c_i64),
                ("host_ag", c_vp), ("dev_gathered", c_vp), ("host_rs_out", c_vp), ("host_rs_in", c_vp),
                ("dev_rs_in", c_vp), ("ag_flags", c_vp), ("ag_landed", c_vp), ("rs_out_flags", c_vp),
                ("rs_in_flags", c_vp), ("rs_landed", c_vp)]


class TraceStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("count", c_i64), ("total_ms", ctypes.c_double),
                ("min_ms", ctypes.c_double), ("max_ms", ctypes.c_double), ("p10_ms", ctypes.c_double),
                ("p50_ms", ctypes.c_double), ("p90_ms", ctypes.c_double)]


# name -> (restype, argtypes)
SIGNATURES = {
    "ep_abi_version": (c_i32, []),
    "ep_status_name": (ctypes.c_char_p, [c_i32]),
    "ep_last_error": (ctypes.c_char_p, []),
    "ep_layout_workspace_bytes": (c_i32, [c_i64, c_i32, c_i32, ctypes.POINTER(c_size)]),
    "ep_dispatch_layout": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                   c_vp, c_size, c_vp]),
    "ep_dispatch_layout_static": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                          c_vp, c_vp]),
    "ep_layout_validate": (c_i32, [c_vp, c_vp]),
    "ep_staging_alloc": (c_i32, [c_i32, c_i64, c_i32, c_i32, c_i32, c_i64, ctypes.POINTER(c_vp)]),
    "ep_staging_free": (c_i32, [c_vp]),
    "ep_staging_ptrs": (c_i32, [c_vp, c_i32, ctypes.POINTER(StagingView)]),
    "ep_staging_set_wait": (c_i32, [c_vp, c_i64, c_i32]),
    "ep_staging_status": (c_i32, [c_vp, c_vp]),
    "ep_staging_set_mode": (c_i32, [c_vp, c_u32, c_i32]),
    "ep_staging_set_inbound": (c_i32, [c_vp, c_i32, ctypes.POINTER(c_i64)]),
    "ep_dispatch": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_vp, c_vp, c_vp, c_i32, c_u32, c_vp]),
    "ep_dispatch_fused": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp,
                                  c_vp, c_size, c_vp, c_i32, c_vp, c_i32, c_u32, c_vp]),
    "ep_combine": (c_i32, [c_vp, c_i32, c_u32, c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_vp, c_i32, c_vp]),
    "ep_round_advance": (c_i32, [c_vp, c_vp]),
    "ep_round_read": (c_i32, [c_vp, ctypes.POINTER(c_u32)]),
    "ep_dispatch_graph": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_vp, c_vp, c_vp]),
    "ep_combine_graph": (c_i32, [c_vp, c_vp, c_vp, c_i64, c_i32, c_i32, c_vp, c_i32, c_vp]),
    "ep_graph_legs_sdma": (c_i32, [c_vp, c_i32]),
    "ep_sim_graph_start": (c_i32, [c_vp, c_i64, c_i64, c_i32, ctypes.POINTER(c_vp)]),
    "ep_sim_graph_wait": (c_i32, [c_vp, c_u32, c_i64]),
    "ep_dense_alloc": (c_i32, [c_i64, c_i32, c_i32, c_i32, c_i32, c_i32, ctypes.POINTER(c_vp)]),
    "ep_dense_free": (c_i32, [c_vp]),
    "ep_dense_get": (c_i32, [c_vp, c_i32, ctypes.POINTER(DenseView)]),
    "ep_dense_set_policy": (c_i32, [c_vp, c_u32, c_i64, c_i32]),
    "ep_dense_status": (c_i32, [c_vp, c_vp]),
    "ep_dense_bytes": (c_i32, [c_vp, ctypes.POINTER(c_i64), ctypes.POINTER(c_i64)]),
    "ep_allgather": (c_i32, [c_vp, c_i32, c_u32, c_vp, c_i64, c_vp]),
    "ep_reducescatter": (c_i32, [c_vp, c_i32, c_u32, c_vp, c_i64, c_i32, c_vp, c_i32, c_vp]),
    "ep_dispatch_layout_local": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp,
                                         c_size, c_vp]),
    "ep_pack": (c_i32, [c_vp, c_i64, c_i32, c_i32, c_vp, c_vp, c_i64, c_vp]),
    "ep_combine_rows": (c_i32, [c_vp, c_i64, c_vp, c_vp, c_i64, c_i32, c_i32, c_vp, c_i32, c_vp]),
    "ep_trace_enable": (c_i32, [c_i32]),
    "ep_trace_read": (c_i32, [ctypes.POINTER(TraceStat), c_i32, ctypes.POINTER(c_i32)]),
    "ep_trace_reset": (c_i32, []),
    "ep_copy_probe": (c_i32, [c_vp, c_vp, c_size, c_vp]),
    "ep_stream_probe": (c_i32, [c_vp, c_vp, c_i64, c_i32, c_i32, c_i32, c_i32, c_vp]),
    "ep_memcpy": (c_i32, [c_vp, c_vp, c_size, c_vp]),
    "ep_pcie_probe": (c_i32, [c_vp, c_vp, c_size, c_i32, ctypes.POINTER(ctypes.c_double)]),
    "ep_sim_peers_start": (c_i32, [c_vp, c_i32, ctypes.POINTER(c_vp)]),
    "ep_sim_peers_post": (c_i32, [c_vp, c_i32, c_u32, c_i64, c_i64]),
    "ep_sim_peers_set_delays": (c_i32, [c_vp, ctypes.POINTER(c_i64), ctypes.POINTER(c_i64)]),
    "ep_sim_dense_start": (c_i32, [c_vp, ctypes.POINTER(c_vp)]),
    "ep_sim_dense_post": (c_i32, [c_vp, c_i32, c_u32, c_i32]),
    "ep_sim_peers_drain": (c_i32, [c_vp, c_i64]),
    "ep_sim_peers_stop": (c_i32, [c_vp]),
}

_lib = None


def load(path: str = LIB_PATH):
    """Load libep.so; raises if it is missing (build it with __graft_entry__.build())."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if lib.ep_abi_version() != ABI_VERSION:
        raise RuntimeError("libep.so ABI version mismatch")
    if path == LIB_PATH:
        _lib = lib
    return lib
