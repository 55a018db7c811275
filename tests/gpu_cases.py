"""Shared inputs and comparisons for the GPU parity tests (HIP path vs. CPU oracle).

Inputs come from the seeded generator (paper_2609_40093_amd.synth) or from simple
routing constructions below; expected values come only from the oracle.
"""
from __future__ import annotations

import dataclasses
import sys

import numpy as np

import oracle
from paper_2609_40093_amd import synth

# combine tolerance on bf16 outputs against the oracle's exact (fp64) sums
TOL_MAX_ABS = 2e-2
TOL_MEAN_ABS = 2e-3


def say(msg: str) -> None:
    """Names the case before a GPU step, flushed, so a crash log still shows it."""
    print(f"[gpu] {msg}", flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class Case:
    name: str
    T: int
    H: int
    E: int
    k: int
    R: int
    x: np.ndarray         # uint16 [T, H]
    topk_idx: np.ndarray  # int32 [T, k]
    topk_w: np.ndarray    # float32 [T, k]
    y: np.ndarray         # uint16 [T*k, H] returned rows in packed order

    @property
    def slots(self):
        return self.T * self.k


def from_config(name: str, **overrides) -> Case:
    cfg = synth.config(name, **overrides)
    inp = synth.make_inputs(cfg)
    return Case(name, cfg.T, cfg.H, cfg.E, cfg.k, cfg.R, inp.x, inp.topk_idx, inp.topk_w, inp.expert_outputs())


def routing(kind: str, T: int, E: int, k: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    if kind == "random":
        if T == 0:
            return np.zeros((0, k), np.int32)
        return np.argsort(rng.random((T, E)), axis=1)[:, :k].astype(np.int32)
    if kind == "roundrobin":
        return (np.arange(T * k) % E).astype(np.int32).reshape(T, k)
    if kind == "firstk":
        return np.tile(np.arange(k, dtype=np.int32), (T, 1))
    if kind == "lastk":
        return np.tile(np.arange(E - k, E, dtype=np.int32)[::-1], (T, 1))
    if kind == "skewed":   # a few hot experts take most rows
        z = rng.standard_normal((T, E)) - 3.0 * np.log1p(np.arange(E))[None, :]
        return np.argsort(-z, axis=1, kind="stable")[:, :k].astype(np.int32)
    raise ValueError(kind)


def make_case(name: str, T: int, H: int, E: int, k: int, R: int, kind: str = "random", seed: int = 0,
              gates: str = "random") -> Case:
    idx = routing(kind, T, E, k, seed)
    ss = np.random.SeedSequence([seed, T, H, E, k])
    sx, sw, sy = ss.spawn(3)
    x = synth.normal_bf16_rows(sx, T, H)
    if gates == "random":
        w = np.random.default_rng(sw).random((T, k)).astype(np.float32) + 0.05
        w = (w / w.sum(axis=1, keepdims=True)).astype(np.float32)
    elif gates == "uniform":
        w = np.full((T, k), 1.0 / k, np.float32)
    else:
        raise ValueError(gates)
    y = synth.normal_bf16_rows(sy, T * k, H)
    return Case(name, T, H, E, k, R, x, idx, w, y)


def bf16_ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance in bf16 steps between two arrays of finite bf16 bit patterns."""
    def ordered(u):
        u = u.astype(np.int32)
        return np.where(u & 0x8000, 0x8000 - u, u)   # monotone integer image of the value
    return np.abs(ordered(a) - ordered(b))


def combine_errors(got_bits: np.ndarray, exact: np.ndarray):
    got = synth.bf16_bits_to_f32(got_bits).astype(np.float64)
    err = np.abs(got - exact)
    return float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0


def oracle_reference(case: Case):
    lay = oracle.layout(case.topk_idx, case.E, case.R)
    assert lay.status == oracle.OK, "oracle rejected the routing"
    packed = oracle.pack(case.x, lay.slot_pos, case.k)
    exact, b16, f32 = oracle.combine(case.y, lay.slot_pos, case.topk_w)
    return lay, packed, exact, b16, f32


def compare_packed_rows(get_rows, x: np.ndarray, row_src: np.ndarray, k: int, rows: int, what: str,
                        chunk: int = 16384) -> None:
    """Every packed row against the pack definition, `chunk` rows at a time: get_rows(r0,
    r1) returns rows [r0, r1) as uint16 [r1-r0, H] (copied from the device or read from a
    host bounce buffer); row p must equal x[row_src[p] // k] bit for bit."""
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        got = get_rows(r0, r1)
        want = oracle.pack_rows(x, row_src, k, np.arange(r0, r1))
        if not np.array_equal(got, want):
            bad = np.nonzero((got != want).any(axis=1))[0]
            raise AssertionError(f"{what}: {len(bad)} packed rows differ in [{r0}, {r1}), first at row {r0 + bad[0]}")


def compare_combine(get_tokens, y: np.ndarray, slot_pos: np.ndarray, topk_w: np.ndarray, what: str,
                    chunk: int = 2048) -> None:
    """Every combined token against the oracle's exact sums, `chunk` tokens at a time:
    get_tokens(t0, t1) returns the bf16 bits of tokens [t0, t1).  Each chunk and the whole
    output must be within max abs TOL_MAX_ABS, and the whole output within mean abs
    TOL_MEAN_ABS."""
    T, k = topk_w.shape
    total, count, worst = 0.0, 0, 0.0
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        slots = slot_pos[t0 * k:t1 * k]
        exact, _, _ = oracle.combine_tokens(y[slots], topk_w[t0:t1])
        got = synth.bf16_bits_to_f32(get_tokens(t0, t1)).astype(np.float64)
        err = np.abs(got - exact)
        worst = max(worst, float(err.max()) if err.size else 0.0)
        total += float(err.sum())
        count += err.size
    mean = total / max(count, 1)
    assert worst <= TOL_MAX_ABS and mean <= TOL_MEAN_ABS, f"{what}: combine error max {worst} mean {mean}"
