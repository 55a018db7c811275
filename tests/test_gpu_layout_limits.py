"""The dispatch layout at the edges of its tile geometry, against the oracle bit for bit.

The multi-tile layout cuts the T*k routing entries into tiles of W waves x `rounds`
rounds x 64 entries and keeps the tiles' count table at most 16K words and 1024 tiles, so
the largest layouts run with the most tiles and many rounds per wave; beyond 8 rounds a
wave no longer keeps its ids and ranks in registers and reads the ids again to write the
positions.  The cases here reach those limits:
  - 1024 tiles of one round (the count table's largest size with 16 experts, which is
    also the most scratch the no-workspace entry point ever needs), through both entry
    points;
  - 1024 tiles of 64 rounds (64M entries: long runs with the ids read twice);
  - 2048 experts (4-wave tiles, at most 8 of them) over 4M entries: thousands of rounds
    per wave.
Routings are seeded: each token row is one of a table of random ordered k-subsets of
the experts, chosen with a skewed (Zipf-like) popularity, so that expert loads differ.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import say
from paper_2609_40093_amd import api

pytestmark = pytest.mark.gpu
DEV = "cuda"
KEYS = ("expert_counts", "expert_offsets", "rank_counts", "rank_offsets", "slot_pos", "row_src")


def table_routing(T: int, E: int, k: int, seed: int, rows: int = 4096) -> np.ndarray:
    """[T, k] int32: each token row one of `rows` random ordered k-subsets of E experts,
    picked with probability proportional to 1 / (rank + 1)."""
    rng = np.random.default_rng(seed)
    table = np.argsort(rng.random((rows, E)), axis=1)[:, :k].astype(np.int32)
    p = 1.0 / np.arange(1, rows + 1)
    pick = rng.choice(rows, size=T, p=p / p.sum())
    return table[pick]


def tiles_of(T: int, k: int, E: int) -> int:
    """Tiles of the layout's geometry, read back from the workspace size it asks for
    (a 256-byte header, then (E + 1) words per tile when there are several)."""
    extra = api.workspace_bytes(T, k, E) - 256
    return extra // (4 * (E + 1)) if extra > 0 else 1


def check_against_oracle(idx: np.ndarray, E: int, R: int, what: str, static_too: bool = False):
    T, k = idx.shape
    say(f"layout limits: {what} (T={T}, k={k}, E={E}, R={R}, tiles={tiles_of(T, k, E)})")
    want = oracle.layout(idx, E, R)
    assert want.status == 0
    idx_d = torch.from_numpy(np.ascontiguousarray(idx)).to(DEV)
    lay = ep.dispatch_layout(idx_d, E, R)
    ep.layout_validate(lay)
    torch.cuda.synchronize()
    for key in KEYS:
        got = getattr(lay, key).cpu().numpy()
        assert np.array_equal(got, getattr(want, key)), f"{what}: {key} differs"
    del lay
    if not static_too:
        return
    # the no-workspace entry point on the same routing, through the C ABI
    lib = api._lib_handle()
    n = T * k
    i32 = dict(dtype=torch.int32, device=DEV)
    outs = [torch.full((E,), -7, **i32), torch.full((E + 1,), -7, **i32), torch.full((R,), -7, **i32),
            torch.full((R + 1,), -7, **i32), torch.full((n,), -7, **i32), torch.full((n,), -7, **i32)]
    status = torch.full((1,), 0x7FFF, dtype=torch.int32, device=DEV)
    say(f"layout limits: {what}, no-workspace entry point")
    assert lib.ep_dispatch_layout_static(api._ptr(idx_d), T, k, E, R, *[api._ptr(t) for t in outs],
                                         api._ptr(status), api._stream_ptr(None)) == 0, lib.ep_last_error()
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for key, t in zip(KEYS, outs):
        assert np.array_equal(t.cpu().numpy(), getattr(want, key)), f"{what} (no workspace): {key} differs"


def test_layout_at_the_tile_cap_one_round():
    T, k, E, R = 1 << 17, 8, 16, 4          # 2^20 entries: 1024 tiles of 16 waves x 1 round
    assert tiles_of(T, k, E) == 1024
    check_against_oracle(table_routing(T, E, k, seed=40), E, R, "1024 tiles, one round", static_too=True)


def test_layout_at_the_tile_cap_long_runs():
    T, k, E, R = 1 << 23, 8, 16, 4          # 2^26 entries: 1024 tiles x 64 rounds (ids read again)
    assert tiles_of(T, k, E) == 1024
    check_against_oracle(table_routing(T, E, k, seed=41), E, R, "1024 tiles, 64 rounds")


def test_layout_widest_experts_thousands_of_rounds():
    T, k, E, R = 1 << 19, 8, 2048, 8        # 2^22 entries over 8 four-wave tiles: 2048 rounds each
    assert tiles_of(T, k, E) == 8
    check_against_oracle(table_routing(T, E, k, seed=42), E, R, "2048 experts, 2048 rounds per wave",
                         static_too=True)


def test_layout_tile_cap_ragged_top3():
    # k = 3 (rows straddle rounds, waves and tiles) with a ragged last tile near the cap
    T, k, E, R = 700001, 3, 40, 4
    check_against_oracle(table_routing(T, E, k, seed=43), E, R, "top-3, ragged, many tiles", static_too=True)
