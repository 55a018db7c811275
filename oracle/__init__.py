"""CPU oracle for MoE expert-parallel dispatch/combine -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package.  The product path (the HIP library and its Python binding) never
imports, links or calls it, and it shares no code with them.

The arithmetic lives in ``ep_oracle.c`` (plain C, built with gcc); this module only
marshals numpy arrays.  Every function follows a passage of the paper (Lee et al.,
"Efficient Expert-Parallel Communication on PCIe-Connected Consumer GPUs"):
  layout  -- Sec. 4.3 grouping of tokens by expert; Sec. 4.5 routing-aware rows
  pack    -- Sec. 2.2 packing of routing-dependent rows into a contiguous region
  combine -- Sec. 4.3 reduction of a token's returned contributions on its owner
  local_layout, block_reduce, pcie_volume -- Sec. 4.2 dense All-Gather / Reduce-Scatter:
             receive-side grouping by local expert, the destination's sum of blocks, and
             the per-GPU PCIe volume of each collective
Pins (tests/test_oracle_*.py): brute force, closed forms, library routines, exact
rational arithmetic; see the module docstrings there.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ep_oracle.c")
LIB_PATH = os.path.join(_HERE, "libep_oracle.so")
CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math", "-fopenmp"]

OK, INVALID_ARG, BAD_ROUTING = 0, 1, 2


def build(src: str = _SRC, out: str = LIB_PATH, extra=()) -> str:
    """Compile the oracle with gcc (always recompiles)."""
    cmd = ["gcc", *CFLAGS, *extra, "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


_lib = None


def _bind(lib):
    i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
    u16p = np.ctypeslib.ndpointer(np.uint16, flags="C_CONTIGUOUS")
    f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
    f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
    vp = ctypes.c_void_p
    lib.ep_oracle_layout.restype = ctypes.c_int
    lib.ep_oracle_layout.argtypes = [i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int32, i32p, i32p, i32p, i32p, i32p, vp]
    lib.ep_oracle_pack.restype = None
    lib.ep_oracle_pack.argtypes = [u16p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, i32p, u16p]
    lib.ep_oracle_combine.restype = None
    lib.ep_oracle_combine.argtypes = [u16p, i32p, f32p, ctypes.c_int64, ctypes.c_int32,
                                      ctypes.c_int32, vp, vp, vp]
    lib.ep_oracle_double_to_bf16_n.restype = None
    lib.ep_oracle_double_to_bf16_n.argtypes = [f64p, ctypes.c_int64, u16p]
    lib.ep_oracle_local_layout.restype = ctypes.c_int
    lib.ep_oracle_local_layout.argtypes = [i32p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, i32p, i32p, i32p, vp]
    lib.ep_oracle_set_threads.restype = ctypes.c_int
    lib.ep_oracle_set_threads.argtypes = [ctypes.c_int]
    lib.ep_oracle_block_reduce.restype = None
    lib.ep_oracle_block_reduce.argtypes = [f64p, ctypes.c_int32, ctypes.c_int64, vp, vp, vp]
    return lib


def load(path: str = LIB_PATH, rebuild_if_missing: bool = True):
    """Load the oracle library (building it first if it is not there)."""
    global _lib
    if path == LIB_PATH and _lib is not None:
        return _lib
    if not os.path.exists(path):
        if not rebuild_if_missing:
            raise FileNotFoundError(path)
        build(out=path)
    lib = _bind(ctypes.CDLL(path))
    if path == LIB_PATH:
        _lib = lib
    return lib


@dataclass
class Layout:
    status: int
    expert_counts: np.ndarray
    expert_offsets: np.ndarray
    rank_counts: np.ndarray
    rank_offsets: np.ndarray
    slot_pos: np.ndarray
    row_src: np.ndarray


def layout(topk_idx: np.ndarray, E: int, R: int, lib=None) -> Layout:
    lib = lib or load()
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    T, k = idx.shape
    n = T * k
    ec = np.zeros(max(E, 1), np.int32)
    eo = np.zeros(max(E, 0) + 1, np.int32)
    rc = np.zeros(max(R, 1), np.int32)
    ro = np.zeros(max(R, 0) + 1, np.int32)
    sp = np.full(max(n, 1), -1, np.int32)
    rs = np.full(max(n, 1), -1, np.int32)
    st = lib.ep_oracle_layout(idx.reshape(-1) if n else np.zeros(1, np.int32), T, k, E, R,
                              ec, eo, rc, ro, sp, rs.ctypes.data)
    return Layout(st, ec[:E], eo[:E + 1], rc[:R], ro[:R + 1], sp[:n], rs[:n])


def pack(x: np.ndarray, slot_pos: np.ndarray, k: int, rows: int = None, lib=None) -> np.ndarray:
    lib = lib or load()
    x = np.ascontiguousarray(x, dtype=np.uint16)
    T, H = x.shape
    rows = T * k if rows is None else rows
    out = np.zeros((max(rows, 1), H), np.uint16)
    if T:
        lib.ep_oracle_pack(x, T, H, k, np.ascontiguousarray(slot_pos, dtype=np.int32), out)
    return out[:rows]


def pack_rows(x: np.ndarray, row_src: np.ndarray, k: int, rows: np.ndarray) -> np.ndarray:
    """The pack definition evaluated at selected packed rows only: row p holds the token
    row x[row_src[p] // k] (for full-size checks where the whole packed buffer is large)."""
    return np.ascontiguousarray(x[np.asarray(row_src)[np.asarray(rows)] // k])


def combine_tokens(y_rows: np.ndarray, topk_w: np.ndarray):
    """combine() for selected tokens: y_rows[i*k + j] is the returned row of slot j of the
    i-th selected token, topk_w [n, k] their gates."""
    n, k = topk_w.shape
    return combine(y_rows, np.arange(n * k, dtype=np.int32), topk_w)


def combine(y: np.ndarray, slot_pos: np.ndarray, topk_w: np.ndarray, lib=None):
    """Returns (exact float64 [T,H], bf16 bits uint16 [T,H], float32 [T,H])."""
    lib = lib or load()
    y = np.ascontiguousarray(y, dtype=np.uint16)
    w = np.ascontiguousarray(topk_w, dtype=np.float32)
    T, k = w.shape
    H = y.shape[1]
    exact = np.zeros((T, H), np.float64)
    b16 = np.zeros((T, H), np.uint16)
    f32 = np.zeros((T, H), np.float32)
    if T and H:
        lib.ep_oracle_combine(y, np.ascontiguousarray(slot_pos, dtype=np.int32).reshape(-1),
                              w.reshape(-1), T, H, k, exact.ctypes.data, b16.ctypes.data,
                              f32.ctypes.data)
    return exact, b16, f32


def set_threads(threads: int, lib=None) -> int:
    """Host threads for pack and combine (1: the plain single-threaded oracle); the outputs
    are the same for any count.  Returns the count in effect."""
    lib = lib or load()
    return int(lib.ep_oracle_set_threads(int(threads)))


def double_to_bf16(v: np.ndarray, lib=None) -> np.ndarray:
    lib = lib or load()
    v = np.ascontiguousarray(v, dtype=np.float64)
    out = np.zeros(v.shape, np.uint16)
    lib.ep_oracle_double_to_bf16_n(v.reshape(-1), v.size, out.reshape(-1))
    return out


def bf16_to_double(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bits to float64 (exact; appends 16 zero bits)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@dataclass
class LocalLayout:
    status: int
    local_counts: np.ndarray
    local_offsets: np.ndarray
    slot_pos: np.ndarray
    row_src: np.ndarray


def local_layout(topk_idx: np.ndarray, E: int, e_lo: int, e_hi: int, lib=None) -> LocalLayout:
    """Grouping of N gathered tokens by the local experts [e_lo, e_hi) (slot_pos -1 elsewhere)."""
    lib = lib or load()
    idx = np.ascontiguousarray(topk_idx, dtype=np.int32)
    N, k = idx.shape
    L = max(e_hi - e_lo, 1)
    lc = np.zeros(L, np.int32)
    lo = np.zeros(L + 1, np.int32)
    sp = np.full(max(N * k, 1), -1, np.int32)
    rs = np.full(max(N * k, 1), -1, np.int32)
    st = lib.ep_oracle_local_layout(idx.reshape(-1) if N else np.zeros(1, np.int32), N, k, E, e_lo, e_hi,
                                    lc, lo, sp, rs.ctypes.data)
    n_local = int(lo[-1]) if st == OK else 0
    return LocalLayout(st, lc, lo, sp[:N * k], rs[:n_local])


def block_reduce(blocks: np.ndarray, lib=None):
    """Sum of R blocks (float64 [R, ...] holding bf16 or float values) in rank order.
    Returns (exact float64, bf16 bits uint16, float32), each shaped like one block."""
    lib = lib or load()
    b = np.ascontiguousarray(blocks, dtype=np.float64)
    R = b.shape[0]
    shape = b.shape[1:]
    n = int(np.prod(shape)) if shape else 1
    exact = np.zeros(n, np.float64)
    b16 = np.zeros(n, np.uint16)
    f32 = np.zeros(n, np.float32)
    if n and R:
        lib.ep_oracle_block_reduce(b.reshape(-1), R, n, exact.ctypes.data, b16.ctypes.data, f32.ctypes.data)
    return exact.reshape(shape), b16.reshape(shape), f32.reshape(shape)


def pcie_volume(collective: str, algorithm: str, N: int, S: float) -> dict:
    """Per-GPU PCIe bytes of the collectives of Sec. 4.2, for N GPUs with shards of S bytes
    (host memory as the only shared medium, every byte crossing PCIe once per hop):
      all_gather ring           each of the N-1 relay steps writes one shard to host memory
                                and reads one back: up (N-1)S, down (N-1)S
      all_gather single_step    upload the own shard once, download the N-1 others:
                                up S, down (N-1)S
      reduce_scatter ring       (N-1)S each way, as the ring All-Gather
      reduce_scatter gpu        upload the N-1 blocks for the other GPUs, download the N-1
                                blocks for this GPU's shard: up (N-1)S, down (N-1)S
      reduce_scatter cpu        upload the N-1 blocks, download one block already summed
                                in host memory: up (N-1)S, down S
    """
    table = {
        ("all_gather", "ring"): ((N - 1) * S, (N - 1) * S),
        ("all_gather", "single_step"): (S, (N - 1) * S),
        ("reduce_scatter", "ring"): ((N - 1) * S, (N - 1) * S),
        ("reduce_scatter", "gpu"): ((N - 1) * S, (N - 1) * S),
        ("reduce_scatter", "cpu"): ((N - 1) * S, S),
    }
    up, down = table[(collective, algorithm)]
    return {"up": up, "down": down, "total": up + down}
