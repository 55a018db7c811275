"""Pins for the CPU oracle: checks against things other than the oracle itself.

Each ``pin_*`` function takes a loaded oracle library (``oracle.load(path)``) and raises
AssertionError when the oracle disagrees with what the paper's definitions and the
mathematics fix:
  * brute force on tiny inputs (Python's comparison sort, exact rational arithmetic),
  * closed forms (round-robin routing, all tokens on the first k experts, identity and
    expert-scaled identity experts with dyadic gates),
  * library routines (numpy stable argsort and fancy indexing, torch's bf16 conversion),
  * hand-derived fixtures under tests/golden/.
The same pins are run against deliberately broken copies of the oracle
(test_oracle_mutants.py) to show that a plausible mistake fails at least one of them.
"""
from __future__ import annotations

import itertools
import os
from fractions import Fraction

import numpy as np

import oracle
from paper_2609_40093_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# ----------------------------------------------------------------------------- helpers

def brute_layout(idx: np.ndarray, E: int, R: int):
    """Layout by definition: rows grouped by expert, token order kept inside a group."""
    flat = [int(v) for v in idx.reshape(-1)]
    n = len(flat)
    order = sorted(range(n), key=lambda i: (flat[i], i))
    slot_pos = [0] * n
    for p, i in enumerate(order):
        slot_pos[i] = p
    counts = [flat.count(e) for e in range(E)]
    offsets = [sum(counts[:e]) for e in range(E + 1)]
    L = E // R
    rank_counts = [sum(counts[r * L:(r + 1) * L]) for r in range(R)]
    rank_offsets = [sum(rank_counts[:r]) for r in range(R + 1)]
    return dict(expert_counts=counts, expert_offsets=offsets, rank_counts=rank_counts,
                rank_offsets=rank_offsets, slot_pos=slot_pos, row_src=order)


def random_routing(rng, T: int, E: int, k: int) -> np.ndarray:
    if T == 0:
        return np.zeros((0, k), np.int32)
    return np.stack([rng.permutation(E)[:k] for _ in range(T)]).astype(np.int32)


def _eq(name, got, want):
    got = np.asarray(got).tolist()
    want = np.asarray(want).tolist()
    assert got == want, f"{name}: oracle {got[:16]} != expected {want[:16]}"


def _check_layout(lib, idx, E, R, want):
    L = oracle.layout(idx, E, R, lib=lib)
    assert L.status == oracle.OK, f"status {L.status}"
    for key in ("expert_counts", "expert_offsets", "rank_counts", "rank_offsets", "slot_pos", "row_src"):
        _eq(key, getattr(L, key), want[key])


def bf16_from_fraction(q: Fraction) -> int:
    """Round an exact rational to bf16, nearest with ties to even, by exact comparisons.

    Independent of the oracle's frexp/nearbyint route: finds the binade by comparing
    with powers of two and the rounding direction by comparing remainders with 1/2."""
    if q == 0:
        return 0
    sign = 0x8000 if q < 0 else 0
    a = abs(q)
    e = 0
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1                                   # now 2^e <= a < 2^(e+1)
    spacing_exp = max(e - 7, -133)               # 8 significant bits; subnormal floor
    m = a / Fraction(2) ** spacing_exp
    n = m.numerator // m.denominator
    rem = m - n
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and n % 2 == 1):
        n += 1
    value = Fraction(n) * Fraction(2) ** spacing_exp
    if value >= Fraction(2) ** 128:
        return sign | 0x7F80
    if value < Fraction(2) ** -126:              # subnormal: fraction field holds n
        return sign | int(n)
    ve = 0
    while value >= Fraction(2) ** (ve + 1):
        ve += 1
    while value < Fraction(2) ** ve:
        ve -= 1
    frac = value / Fraction(2) ** ve - 1         # in [0, 1), multiple of 2^-7
    return sign | ((ve + 127) << 7) | int(frac * 128)


def bf16_fraction(b: int) -> Fraction:
    """Exact value of a finite bf16 bit pattern from its fields."""
    s = -1 if b & 0x8000 else 1
    ex = (b >> 7) & 0xFF
    fr = b & 0x7F
    assert ex != 0xFF
    if ex == 0:
        return s * Fraction(fr) * Fraction(2) ** -133
    return s * (1 + Fraction(fr, 128)) * Fraction(2) ** (ex - 127)


def f32_fraction(f) -> Fraction:
    return Fraction(float(np.float32(f)))


# --------------------------------------------------------------------------- layout pins

def pin_layout_golden(lib):
    """Hand-worked example in the setting of the AG/RS pattern figure (Sec. 2.1)."""
    d = {}
    for line in open(os.path.join(GOLDEN, "layout_agrs_example.txt")):
        if line.startswith("#") or ":" not in line:
            continue
        key, vals = line.split(":", 1)
        d[key.strip()] = [int(v) for v in vals.split()]
    T, k, E, R = d["T"][0], d["k"][0], d["E"][0], d["R"][0]
    idx = np.array(d["topk_idx"], np.int32).reshape(T, k)
    _check_layout(lib, idx, E, R, d)


def pin_layout_bruteforce(lib):
    """Random tiny routings and exhaustive tiny cases against Python's stable sort."""
    rng = np.random.default_rng(1234)
    for _ in range(300):
        E = int(rng.choice([1, 2, 3, 4, 6, 8]))
        R = int(rng.choice([r for r in (1, 2, 3, 4, 8) if E % r == 0]))
        k = int(rng.integers(1, min(E, 3) + 1))
        T = int(rng.integers(0, 13))
        idx = random_routing(rng, T, E, k)
        _check_layout(lib, idx, E, R, brute_layout(idx, E, R))
    # every routing of 2 tokens over 3 experts, top-2 (36 cases), R in {1, 3}
    rows = list(itertools.permutations(range(3), 2))
    for r0, r1 in itertools.product(rows, rows):
        idx = np.array([r0, r1], np.int32)
        for R in (1, 3):
            _check_layout(lib, idx, 3, R, brute_layout(idx, 3, R))
    # every routing of 3 tokens over 4 experts, top-1 (64 cases), R in {1, 2, 4}
    for combo in itertools.product(range(4), repeat=3):
        idx = np.array(combo, np.int32).reshape(3, 1)
        for R in (1, 2, 4):
            _check_layout(lib, idx, 4, R, brute_layout(idx, 4, R))


def pin_layout_closed_forms(lib):
    """Round-robin routing and all-tokens-on-the-first-k-experts have closed forms."""
    for (T, k, E, R) in [(12, 2, 8, 4), (64, 8, 16, 8), (7, 3, 3, 1), (96, 8, 256, 8), (5, 1, 5, 5)]:
        n = T * k
        if n % E:
            continue
        idx = (np.arange(n) % E).astype(np.int32).reshape(T, k)      # idx[t][j] = (t*k+j) mod E
        i = np.arange(n)
        per = n // E
        L = oracle.layout(idx, E, R, lib=lib)
        _eq("rr counts", L.expert_counts, [per] * E)
        _eq("rr offsets", L.expert_offsets, [per * e for e in range(E + 1)])
        _eq("rr slot_pos", L.slot_pos, (i % E) * per + i // E)
        _eq("rr rank_offsets", L.rank_offsets, [per * (E // R) * r for r in range(R + 1)])
    for (T, k, E, R) in [(10, 3, 8, 4), (33, 8, 32, 8), (1, 4, 4, 2)]:
        idx = np.tile(np.arange(k, dtype=np.int32), (T, 1))          # every token -> 0..k-1
        L = oracle.layout(idx, E, R, lib=lib)
        _eq("firstk counts", L.expert_counts, [T] * k + [0] * (E - k))
        t, j = np.divmod(np.arange(T * k), k)
        _eq("firstk slot_pos", L.slot_pos, j * T + t)
        # reversed slot order: slot j -> expert k-1-j; the group of expert e is still token order
        L2 = oracle.layout(idx[:, ::-1].copy(), E, R, lib=lib)
        _eq("firstk reversed slot_pos", L2.slot_pos, (k - 1 - j) * T + t)


def pin_layout_argsort(lib):
    """The synthetic workloads' routing against numpy's stable argsort and bincount."""
    for name in ("tiny", "coarse", "fine", "decode"):
        inp = synth.make_inputs(synth.config(name))
        c = inp.cfg
        flat = inp.topk_idx.reshape(-1)
        L = oracle.layout(inp.topk_idx, c.E, c.R, lib=lib)
        assert L.status == oracle.OK
        order = np.argsort(flat, kind="stable")
        _eq(f"{name} row_src", L.row_src, order)
        inv = np.empty_like(order)
        inv[order] = np.arange(order.size)
        _eq(f"{name} slot_pos", L.slot_pos, inv)
        cnt = np.bincount(flat, minlength=c.E)
        _eq(f"{name} counts", L.expert_counts, cnt)
        _eq(f"{name} rank_counts", L.rank_counts, cnt.reshape(c.R, -1).sum(axis=1))


def pin_layout_invariants(lib):
    """Sum of counts, permutation, monotone offsets, stability, rank = expert boundaries."""
    rng = np.random.default_rng(7)
    for (T, k, E, R) in [(1000, 8, 128, 8), (333, 2, 8, 4), (1, 1, 1, 1), (50, 16, 16, 2)]:
        idx = random_routing(rng, T, E, k)
        L = oracle.layout(idx, E, R, lib=lib)
        n = T * k
        assert int(L.expert_counts.sum()) == n
        assert sorted(L.slot_pos.tolist()) == list(range(n))
        assert np.all(np.diff(L.expert_offsets) >= 0) and L.expert_offsets[-1] == n
        assert (L.rank_offsets == L.expert_offsets[::E // R]).all()
        flat = idx.reshape(-1)
        grp = flat[L.row_src]
        assert np.all(np.diff(grp) >= 0), "groups not in expert order"
        same = np.diff(grp) == 0
        assert np.all(np.diff(L.row_src)[same] > 0), "token order not kept inside a group"
        assert (L.slot_pos[L.row_src] == np.arange(n)).all()


def pin_layout_validation(lib):
    """Bad ids and repeated experts in a token row are rejected; bad sizes too."""
    ok = np.array([[0, 1], [2, 3]], np.int32)
    assert oracle.layout(ok, 4, 2, lib=lib).status == oracle.OK
    assert oracle.layout(np.array([[0, 4], [2, 3]], np.int32), 4, 2, lib=lib).status == oracle.BAD_ROUTING
    assert oracle.layout(np.array([[0, -1], [2, 3]], np.int32), 4, 2, lib=lib).status == oracle.BAD_ROUTING
    assert oracle.layout(np.array([[1, 1], [2, 3]], np.int32), 4, 2, lib=lib).status == oracle.BAD_ROUTING
    assert oracle.layout(np.array([[0, 1, 2], [3, 2, 3]], np.int32), 4, 2, lib=lib).status == oracle.BAD_ROUTING
    assert oracle.layout(ok, 4, 3, lib=lib).status == oracle.INVALID_ARG     # E % R != 0
    assert oracle.layout(np.zeros((2, 5), np.int32), 4, 2, lib=lib).status == oracle.INVALID_ARG  # k > E
    L = oracle.layout(np.zeros((0, 2), np.int32), 4, 2, lib=lib)
    assert L.status == oracle.OK and L.expert_counts.tolist() == [0] * 4
    assert L.expert_offsets.tolist() == [0] * 5 and L.rank_offsets.tolist() == [0, 0, 0]


# ----------------------------------------------------------------------------- pack pin

def pin_pack(lib):
    """packed[p] == x[row_src[p] // k] byte for byte (numpy fancy indexing)."""
    rng = np.random.default_rng(3)
    for (T, H, E, k, R) in [(37, 24, 8, 3, 4), (128, 1024, 16, 2, 4), (5, 8, 5, 5, 1), (1, 16, 1, 1, 1)]:
        idx = random_routing(rng, T, E, k)
        b = brute_layout(idx, E, R)
        x = rng.integers(0, 1 << 16, size=(T, H), dtype=np.uint16)
        packed = oracle.pack(x, np.array(b["slot_pos"], np.int32), k, lib=lib)
        want = x[np.array(b["row_src"]) // k]
        assert packed.tobytes() == want.tobytes(), "packed rows differ"
        rows = np.arange(T * k)[::3]
        assert oracle.pack_rows(x, np.array(b["row_src"]), k, rows).tobytes() == packed[rows].tobytes()


# --------------------------------------------------------------------------- combine pins

def _combine_case(rng, T, H, E, k):
    idx = random_routing(rng, T, E, k)
    b = brute_layout(idx, E, 1)
    return np.array(b["slot_pos"], np.int32), np.array(b["row_src"], np.int64), idx


def pin_combine_fraction(lib):
    """Exact rational sums on tiny inputs: the double result is within the bound of k
    roundings, and the bf16 output is the nearest-even rounding of that double."""
    rng = np.random.default_rng(11)
    for _ in range(40):
        T, H, E = int(rng.integers(1, 5)), int(rng.integers(1, 9)), 8
        k = int(rng.integers(1, 5))
        slot_pos, _, _ = _combine_case(rng, T, H, E, k)
        # bf16 inputs with wide exponents, signs and zeros; gates are arbitrary floats
        y = rng.integers(0, 1 << 16, size=(T * k, H), dtype=np.uint16)
        y[(y & 0x7F80) == 0x7F80] &= 0xBFFF                      # no inf/NaN
        y &= np.uint16(0xCFFF)                                  # keep exponents moderate
        w = rng.standard_normal((T, k)).astype(np.float32)
        exact, b16, _ = oracle.combine(y, slot_pos, w, lib=lib)
        for t in range(T):
            for h in range(H):
                terms = [f32_fraction(w[t, j]) * bf16_fraction(int(y[slot_pos[t * k + j], h]))
                         for j in range(k)]
                q = sum(terms, Fraction(0))
                bound = Fraction(k) * Fraction(2) ** -52 * sum(abs(x) for x in terms)
                assert abs(Fraction(float(exact[t, h])) - q) <= bound, "double sum off"
                assert int(b16[t, h]) == bf16_from_fraction(Fraction(float(exact[t, h]))), \
                    f"bf16 rounding of {float(exact[t, h])!r}"


def pin_combine_inverse_permutation(lib):
    """k = 1 with gate 1 returns each token's row unchanged, bit for bit."""
    rng = np.random.default_rng(5)
    T, H, E = 50, 40, 6
    slot_pos, _, _ = _combine_case(rng, T, H, E, 1)
    y = rng.integers(0, 1 << 16, size=(T, H), dtype=np.uint16)
    y[(y & 0x7F80) == 0x7F80] &= 0xBFFF
    _, b16, _ = oracle.combine(y, slot_pos, np.ones((T, 1), np.float32), lib=lib)
    assert b16.tobytes() == y[slot_pos].tobytes()
    # the per-token form gives the same rows
    _, b16_tok, _ = oracle.combine_tokens(y[slot_pos[::2]], np.ones((len(slot_pos[::2]), 1), np.float32))
    assert b16_tok.tobytes() == b16[::2].tobytes()


def pin_combine_identity(lib):
    """Identity experts (y = packed x): dyadic gates summing to 1 give x exactly (bf16 and
    float outputs); the workloads' softmax gates give x within 1e-2 relative."""
    rng = np.random.default_rng(9)
    for (T, H, E, k, gates) in [(40, 32, 8, 2, [0.5, 0.5]), (30, 16, 16, 4, [0.5, 0.25, 0.125, 0.125]),
                                (20, 8, 4, 3, [0.25, 0.5, 0.25])]:
        slot_pos, row_src, _ = _combine_case(rng, T, H, E, k)
        x = synth.normal_bf16_rows(np.random.SeedSequence(T), T, H)
        y = x[row_src // k]                                     # what an identity expert returns
        w = np.tile(np.array(gates, np.float32), (T, 1))
        _, b16, f32 = oracle.combine(y, slot_pos, w, lib=lib)
        assert b16.tobytes() == x.tobytes()
        assert (f32 == synth.bf16_bits_to_f32(x)).all()
    inp = synth.make_inputs(synth.config("tiny"))
    c = inp.cfg
    b = brute_layout(inp.topk_idx, c.E, c.R)
    y = inp.x[np.array(b["row_src"]) // c.k]
    exact, _, _ = oracle.combine(y, np.array(b["slot_pos"], np.int32), inp.topk_w, lib=lib)
    xf = synth.bf16_bits_to_f32(inp.x).astype(np.float64)
    assert np.all(np.abs(exact - xf) <= 1e-2 * np.abs(xf) + 1e-30)


def pin_combine_scaled_identity(lib):
    """Expert e returns 2^(e mod 4) * x; with dyadic gates the result is exactly
    x * sum_j w_j 2^(e_j mod 4): a slot read from the wrong row or the wrong expert shows."""
    rng = np.random.default_rng(13)
    for (T, H, E, k, gates) in [(64, 16, 16, 2, [0.75, 0.25]), (16, 8, 32, 4, [0.5, 0.25, 0.125, 0.125])]:
        slot_pos, row_src, idx = _combine_case(rng, T, H, E, k)
        x = synth.normal_bf16_rows(np.random.SeedSequence(H), T, H)
        xf = synth.bf16_bits_to_f32(x).astype(np.float64)
        flat = idx.reshape(-1)
        scale = 2.0 ** (flat[row_src] % 4)                     # expert of packed row p
        yf = xf[row_src // k] * scale[:, None]
        y = (yf.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)   # exact: power-of-2 scaling
        w = np.tile(np.array(gates, np.float32), (T, 1))
        want = xf * (w.astype(np.float64) * 2.0 ** (idx % 4)).sum(axis=1)[:, None]
        exact, _, f32 = oracle.combine(y, slot_pos, w, lib=lib)
        assert (exact == want).all()
        assert (f32.astype(np.float64) == want).all()


# ------------------------------------------------------------------------------ bf16 pins

def pin_bf16_golden(lib):
    for line in open(os.path.join(GOLDEN, "bf16_rounding.txt")):
        if line.startswith("#") or not line.strip():
            continue
        a, b = line.split()[:2]
        v = float(a) if "inf" in a else float.fromhex(a)
        got = int(oracle.double_to_bf16(np.array([v]), lib=lib)[0])
        assert got == int(b, 16), f"{a}: {got:#06x} != {b}"


def pin_bf16_torch(lib):
    """float32 -> bf16 against torch's conversion (round to nearest even) on CPU."""
    import torch
    rng = np.random.default_rng(17)
    bits = rng.integers(0, 1 << 32, size=200000, dtype=np.uint64).astype(np.uint32)
    bits[:1000] = (bits[:1000] & 0xFFFF0000) | 0x8000          # exact ties
    bits[1000:2000] &= 0x807FFFFF                              # subnormals
    v = bits.view(np.float32)
    v = v[np.isfinite(v)]
    want = torch.from_numpy(v.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.double_to_bf16(v.astype(np.float64), lib=lib)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, f"{bad.size} mismatches, first {v[bad[0]]!r}"
    got_nan = oracle.double_to_bf16(np.array([np.nan, -np.nan]), lib=lib)
    assert all((int(g) & 0x7F80) == 0x7F80 and (int(g) & 0x7F) for g in got_nan)


# ------------------------------------------------------------ dense All-Gather / Reduce-Scatter

def brute_local_layout(idx: np.ndarray, e_lo: int, e_hi: int):
    """Grouping by definition: the slots naming a local expert, ordered by (expert, slot)."""
    flat = [int(v) for v in idx.reshape(-1)]
    local = [i for i in range(len(flat)) if e_lo <= flat[i] < e_hi]
    order = sorted(local, key=lambda i: (flat[i], i))
    slot_pos = [-1] * len(flat)
    for p, i in enumerate(order):
        slot_pos[i] = p
    counts = [flat.count(e) for e in range(e_lo, e_hi)]
    offsets = [sum(counts[:l]) for l in range(e_hi - e_lo + 1)]
    return dict(local_counts=counts, local_offsets=offsets, slot_pos=slot_pos, row_src=order)


def pin_local_layout_bruteforce(lib):
    rng = np.random.default_rng(41)
    for N, E, k in [(1, 4, 2), (9, 6, 3), (40, 16, 4), (64, 8, 8), (0, 4, 1)]:
        idx = random_routing(rng, N, E, k)
        for e_lo, e_hi in [(0, E), (0, 1), (E - 1, E), (E // 4, E // 2 + 1)]:
            if e_lo >= e_hi:
                continue
            got = oracle.local_layout(idx, E, e_lo, e_hi, lib=lib)
            assert got.status == oracle.OK
            want = brute_local_layout(idx, e_lo, e_hi)
            for key, val in want.items():
                _eq(f"local {key} N={N} window=[{e_lo},{e_hi})", getattr(got, key), val)


def pin_local_layout_window_of_global(lib):
    """Inside its window, the local grouping is the global one shifted by the window's first
    offset (the global layout is pinned on its own)."""
    cfg = synth.config("fine")
    idx = synth.make_inputs(cfg).topk_idx[:2000]
    g = oracle.layout(idx, cfg.E, cfg.R, lib=lib)
    L = cfg.E // cfg.R
    flat = idx.reshape(-1)
    for r in range(cfg.R):
        loc = oracle.local_layout(idx, cfg.E, r * L, (r + 1) * L, lib=lib)
        inside = (flat >= r * L) & (flat < (r + 1) * L)
        _eq("local slot_pos", loc.slot_pos[inside], g.slot_pos[inside] - g.expert_offsets[r * L])
        assert np.all(loc.slot_pos[~inside] == -1)
        _eq("local counts", loc.local_counts, g.expert_counts[r * L:(r + 1) * L])


def pin_local_layout_validation(lib):
    idx = np.array([[0, 1], [2, 3]], np.int32)
    for e_lo, e_hi in [(2, 2), (3, 1), (-1, 2), (0, 5)]:
        assert oracle.local_layout(idx, 4, e_lo, e_hi, lib=lib).status == oracle.INVALID_ARG
    assert oracle.local_layout(np.array([[0, 4]], np.int32), 4, 0, 2, lib=lib).status == oracle.BAD_ROUTING
    assert oracle.local_layout(np.array([[3, 3]], np.int32), 4, 0, 2, lib=lib).status == oracle.BAD_ROUTING


def pin_partials_sum_to_combine(lib):
    """Every rank's partial block over its own experts, summed over ranks, is the combine of
    the routing-aware path (exact: dyadic gates and small-integer rows)."""
    rng = np.random.default_rng(43)
    N, H, E, k, R = 50, 12, 16, 4, 4
    idx = random_routing(rng, N, E, k)
    w = (rng.integers(1, 8, size=(N, k)) / 8.0).astype(np.float32)
    g = oracle.layout(idx, E, R, lib=lib)
    vals = rng.integers(-64, 64, size=(N * k, H)).astype(np.float32)
    y = (vals.view(np.uint32) >> 16).astype(np.uint16)        # exact bf16 of small integers
    full, _, _ = oracle.combine(y, g.slot_pos, w, lib=lib)
    L = E // R
    total = np.zeros_like(full)
    for r in range(R):
        loc = oracle.local_layout(idx, E, r * L, (r + 1) * L, lib=lib)
        y_loc = y[g.slot_pos[loc.row_src]] if loc.row_src.size else np.zeros((0, H), np.uint16)
        part, _, _ = oracle.combine(np.ascontiguousarray(y_loc) if y_loc.size else np.zeros((1, H), np.uint16),
                                    loc.slot_pos, w, lib=lib)
        total += part
    _eq("sum of partial blocks", total, full)


def pin_block_reduce_fraction(lib):
    """Exact rational sums of bf16 blocks, rounded by the independent ties-to-even helper."""
    rng = np.random.default_rng(44)
    R, n = 5, 300
    # sign and fraction random, exponents within 2^-20..2^20: five 8-bit significands
    # spanning 40 binades sum exactly in double, so one rounding to bf16 is compared
    sign = rng.integers(0, 2, size=(R, n), dtype=np.uint32) << 15
    expo = rng.integers(127 - 20, 127 + 21, size=(R, n), dtype=np.uint32) << 7
    frac = rng.integers(0, 128, size=(R, n), dtype=np.uint32)
    bits = (sign | expo | frac).astype(np.uint16)
    vals = oracle.bf16_to_double(bits)
    exact, b16, _ = oracle.block_reduce(vals, lib=lib)
    for i in range(n):
        q = sum((bf16_fraction(int(bits[d, i])) for d in range(R)), Fraction(0))
        assert exact[i] == float(q) or abs(Fraction(exact[i]) - q) <= abs(q) * Fraction(1, 1 << 50), i
        assert int(b16[i]) == bf16_from_fraction(q), f"block_reduce bf16 at {i}"
    ones = np.ones((7, 3), np.float64) * 0.75
    _eq("seven equal blocks", oracle.block_reduce(ones, lib=lib)[0], np.full(3, 5.25))


def pin_pcie_volume_golden(lib):
    del lib
    for line in open(os.path.join(GOLDEN, "pcie_volume.txt")):
        line = line.split("#")[0].split()
        if not line:
            continue
        coll, alg, N, total = line[0], line[1], int(line[2]), int(line[3])
        got = oracle.pcie_volume(coll, alg, N, 1.0)["total"]
        assert got == total, f"{coll} {alg} N={N}: model {got} != paper {total}"


ALL_PINS = [pin_layout_golden, pin_layout_bruteforce, pin_layout_closed_forms, pin_layout_argsort,
            pin_layout_invariants, pin_layout_validation, pin_pack, pin_combine_fraction,
            pin_combine_inverse_permutation, pin_combine_identity, pin_combine_scaled_identity,
            pin_bf16_golden, pin_bf16_torch,
            pin_local_layout_bruteforce, pin_local_layout_window_of_global, pin_local_layout_validation,
            pin_partials_sum_to_combine, pin_block_reduce_fraction, pin_pcie_volume_golden]
