"""Seeded synthetic MoE-layer inputs for one rank of a simulated expert-parallel group.

This module only *generates data*: token activations, top-k routing with gate weights,
and the expert outputs that the simulated peer ranks send back.  It holds none of the
dispatch/combine arithmetic, so both the GPU path and the CPU oracle can be fed from it.

Shapes follow the MoE layer of the paper's background section (Sec. 2.1: a router picks
k of E experts per token; experts are split over R devices under EP).  The five named
workloads stand in for the paper's model-level runs (Qwen3-30B-A3B-shaped and
DeepSeek-V3-shaped routing); all values are synthetic.

Recipe (numpy PCG64, ``SeedSequence(seed).spawn(4)``):
  stream 0 -> token activations x, stream 1 -> router logits, stream 2 -> per-expert
  bias / Zipf rank permutation, stream 3 -> returned expert outputs y.
  Large arrays are drawn in fixed row blocks, each block with its own spawned seed, so
  the result does not depend on how many threads draw them.
  bf16 values are float32 normals rounded to the nearest bf16 value, ties to even (the
  samples are finite, so the rounding never reaches infinity or NaN).
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

__all__ = ["LayerConfig", "LayerInputs", "CONFIGS", "config", "make_inputs", "normal_bf16_rows",
           "bf16_bits_to_f32"]

# elements per generation block (fixed: the block partition is part of the recipe)
_BLOCK_ELEMS = 1 << 22


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    name: str
    T: int            # tokens owned by this rank
    H: int            # hidden size (bf16 elements per token row)
    E: int            # experts in the layer
    k: int            # experts per token
    R: int            # ranks in the simulated EP group (experts placed contiguously, E/R per rank)
    gate: str         # "softmax" (softmax over the selected logits) or "sigmoid" (sigmoid, renormalised)
    bias: str         # "none", "normal" (b_e ~ N(0, bias_scale)), or "zipf" (b_e = -s ln rho_e)
    bias_scale: float = 0.0
    staging: tuple = ("hbm",)
    seed: int = 0

    @property
    def slots(self) -> int:
        return self.T * self.k

    @property
    def payload_bytes(self) -> int:
        """Token payload of one dispatch (or one combine): every (token, slot) row, bf16."""
        return self.T * self.k * self.H * 2


CONFIGS = {
    "tiny": LayerConfig("tiny", 128, 1024, 16, 2, 4, "softmax", "none", 0.0, ("hbm",)),
    "coarse": LayerConfig("coarse", 4096, 4096, 8, 2, 4, "softmax", "normal", 0.5, ("hbm", "pinned")),
    "fine": LayerConfig("fine", 8192, 2048, 128, 8, 8, "softmax", "zipf", 1.1, ("pinned",)),
    "decode": LayerConfig("decode", 256, 7168, 256, 8, 8, "sigmoid", "none", 0.0, ("pinned",)),
    "prefill": LayerConfig("prefill", 32768, 7168, 256, 8, 8, "sigmoid", "zipf", 1.2, ("hbm", "pinned")),
}


def config(name: str, **overrides) -> LayerConfig:
    base = CONFIGS[name]
    return dataclasses.replace(base, **overrides) if overrides else base


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal_bf16_rows(ss: np.random.SeedSequence, rows: int, cols: int,
                     row_begin: int = 0, row_end: Optional[int] = None) -> np.ndarray:
    """bf16 bit patterns (uint16) of N(0,1) samples, shape [row_end-row_begin, cols].

    Rows are drawn in blocks of ``max(1, 2**22 // cols)`` rows; block b is drawn from the
    child seed with spawn key ``ss.spawn_key + (b,)`` (what ``ss.spawn`` would hand out,
    built directly so that ``ss`` is never mutated).  Any row range can therefore be
    regenerated, bit-identically, without drawing the rest.
    """
    if row_end is None:
        row_end = rows
    out = np.empty((row_end - row_begin, cols), dtype=np.uint16)
    if rows == 0 or cols == 0 or row_end <= row_begin:
        return out
    block = max(1, _BLOCK_ELEMS // cols)
    first, last = row_begin // block, (row_end - 1) // block

    def draw(b: int) -> None:
        r0, r1 = b * block, min(rows, (b + 1) * block)
        buf = np.empty((r1 - r0, cols), dtype=np.float32)
        child = np.random.SeedSequence(ss.entropy, spawn_key=tuple(ss.spawn_key) + (b,),
                                       pool_size=ss.pool_size)
        np.random.default_rng(child).standard_normal(out=buf, dtype=np.float32)
        lo, hi = max(r0, row_begin), min(r1, row_end)
        bits = buf[lo - r0:hi - r0].view(np.uint32)
        bits = bits + (np.uint32(0x7FFF) + ((bits >> np.uint32(16)) & np.uint32(1)))
        out[lo - row_begin:hi - row_begin] = (bits >> np.uint32(16)).astype(np.uint16)

    blocks = range(first, last + 1)
    if len(blocks) == 1:
        draw(first)
    else:
        with ThreadPoolExecutor(_workers()) as ex:
            list(ex.map(draw, blocks))
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 values (exact)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)


def _routing(cfg: LayerConfig, ss_logits, ss_bias):
    T, E, k = cfg.T, cfg.E, cfg.k
    logits = np.random.default_rng(ss_logits).standard_normal((T, E), dtype=np.float32).astype(np.float64)
    rng_b = np.random.default_rng(ss_bias)
    if cfg.bias == "none":
        bias = np.zeros(E)
    elif cfg.bias == "normal":
        bias = rng_b.normal(0.0, cfg.bias_scale, size=E)
    elif cfg.bias == "zipf":
        rho = rng_b.permutation(E) + 1.0              # Zipf rank of each expert
        bias = -cfg.bias_scale * np.log(rho)          # exp(bias) proportional to rho**-s
    else:
        raise ValueError(f"unknown bias kind {cfg.bias!r}")
    z = logits + bias[None, :]
    idx = np.argsort(-z, axis=1, kind="stable")[:, :k]     # ties -> lower expert id; slot j by score
    zs = np.take_along_axis(z, idx, axis=1)
    if cfg.gate == "softmax":
        g = np.exp(zs - zs.max(axis=1, keepdims=True))
    elif cfg.gate == "sigmoid":
        g = 1.0 / (1.0 + np.exp(-zs))
    else:
        raise ValueError(f"unknown gate kind {cfg.gate!r}")
    g = g / g.sum(axis=1, keepdims=True)
    return idx.astype(np.int32), g.astype(np.float32)


@dataclasses.dataclass
class LayerInputs:
    cfg: LayerConfig
    x: np.ndarray          # uint16 [T, H] bf16 bits: this rank's token activations
    topk_idx: np.ndarray   # int32 [T, k]: selected experts, slot j in descending router score
    topk_w: np.ndarray     # float32 [T, k]: gate weights (sum to 1 per token)
    _ss_y: np.random.SeedSequence = dataclasses.field(repr=False, default=None)

    def expert_outputs(self, row_begin: int = 0, row_end: Optional[int] = None) -> np.ndarray:
        """Returned expert outputs y, uint16 [T*k, H] in the packed (slot-position) order.

        Row p is the output the owning peer computed for packed row p.  The peers' expert
        computation is not simulated; rows are independent N(0,1) bf16 samples.
        """
        return normal_bf16_rows(self._ss_y, self.cfg.slots, self.cfg.H, row_begin, row_end)


def make_inputs(cfg: LayerConfig) -> LayerInputs:
    ss_x, ss_logits, ss_bias, ss_y = np.random.SeedSequence(cfg.seed).spawn(4)
    x = normal_bf16_rows(ss_x, cfg.T, cfg.H)
    idx, w = _routing(cfg, ss_logits, ss_bias)
    return LayerInputs(cfg, x, idx, w, ss_y)


def expected_distinct_ranks(topk_idx: np.ndarray, E: int, R: int) -> float:
    """Mean number of distinct destination ranks per token (a reported statistic)."""
    if topk_idx.size == 0:
        return 0.0
    L = E // R
    ranks = np.sort(topk_idx // L, axis=1)
    return float(1 + (np.diff(ranks, axis=1) != 0).sum(axis=1).mean())


def describe(cfg: LayerConfig) -> str:
    return (f"{cfg.name}: T={cfg.T} H={cfg.H} E={cfg.E} k={cfg.k} R={cfg.R} gate={cfg.gate} "
            f"bias={cfg.bias}({cfg.bias_scale}) payload={cfg.payload_bytes / 1e6:.1f} MB")


if __name__ == "__main__":  # pragma: no cover
    for name in CONFIGS:
        c = CONFIGS[name]
        if c.T * c.H > 1 << 26:
            print(describe(c), "(skipped)")
            continue
        inp = make_inputs(c)
        cnt = np.bincount(inp.topk_idx.ravel(), minlength=c.E)
        print(describe(c), "counts min/max", cnt.min(), cnt.max(),
              "ranks/token", round(expected_distinct_ranks(inp.topk_idx, c.E, c.R), 2))
