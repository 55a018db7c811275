"""Plants plausible mistakes in copies of the oracle (on the CPU) and checks that every
one of them fails at least one pin: the pins are strong enough to trust the oracle.

Each mutant is a textual edit of ep_oracle.c compiled to a temporary library; the real
oracle is untouched.  Mutations are chosen to stay inside the buffers they write.
"""
import os

import pytest

import oracle
import oracle_pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "ep_oracle.c")

MUTANTS = {
    "unstable_placement": ("for (int64_t i = 0; i < n; ++i) {\n        int32_t e = topk_idx[i];",
                           "for (int64_t i = n - 1; i >= 0; --i) {\n        int32_t e = topk_idx[i];"),
    "cursor_not_advanced": ("        cursor[e] += 1;\n", "\n"),
    "rank_offset_index": ("rank_offsets[r] = expert_offsets[r * L];", "rank_offsets[r] = expert_offsets[r];"),
    "rank_strided_experts": ("for (int32_t e = r * L; e < (r + 1) * L; ++e)",
                             "for (int32_t e = r; e < E; e += R)"),
    "no_duplicate_check": ("if (topk_idx[t * k + jj] == e)\n                    status", "if (0)\n                    status"),
    "local_no_duplicate_check": ("if (topk_idx[t * k + jj] == e)\n                    return", "if (0)\n                    return"),
    "pack_wrong_token": ("x + t * (int64_t)H, row_bytes", "x + ((t * k + j) % T) * (int64_t)H, row_bytes"),
    "combine_drops_first_slot": ("for (int32_t j = 0; j < k; ++j) {\n            if (slot_pos[t * k + j] < 0)",
                                 "for (int32_t j = 1; j < k; ++j) {\n            if (slot_pos[t * k + j] < 0)"),
    "combine_gate_transposed": ("double w = (double)topk_w[t * k + j];", "double w = (double)topk_w[j * T + t];"),
    "combine_ignores_slot_pos": ("y + (int64_t)slot_pos[t * k + j] * H", "y + (t * k + j) * (int64_t)H"),
    "combine_float_accumulator": ("acc[h] = acc[h] + w * ep_oracle_bf16_to_double(row[h]);",
                                  "acc[h] = (float)(acc[h] + w * ep_oracle_bf16_to_double(row[h]));"),
    "round_ties_away": ("double n = nearbyint(ldexp(a, -qexp));", "double n = round(ldexp(a, -qexp));"),
    "round_truncate": ("double n = nearbyint(ldexp(a, -qexp));", "double n = trunc(ldexp(a, -qexp));"),
    "subnormal_spacing": ("if (qexp < -133)\n        qexp = -133;", "if (qexp < -126)\n        qexp = -126;"),
    "widen_shift": ("uint32_t bits = (uint32_t)b << 16;", "uint32_t bits = (uint32_t)b << 15;"),
    "local_count_shifted": ("local_counts[e - e_lo] += 1;", "local_counts[(e - e_lo + 1) % L] += 1;"),
    "local_unstable_placement": ("for (int64_t i = 0; i < N * k; ++i) {\n        int32_t e = topk_idx[i];\n        if (e < e_lo",
                                 "for (int64_t i = N * k - 1; i >= 0; --i) {\n        int32_t e = topk_idx[i];\n        if (e < e_lo"),
    "local_window_ignored": ("if (e >= e_lo && e < e_hi)\n            local_counts", "if (e >= e_lo && e < e_hi && e != e_lo)\n            local_counts"),
    "block_reduce_drops_last": ("for (int32_t d = 0; d < R; ++d)   /* blocks", "for (int32_t d = 0; d + 1 < R; ++d)   /* blocks"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mut = tmp_path / "ep_oracle.c"
    mut.write_text(src.replace(old, new))
    (tmp_path / "ep_oracle.h").write_text(open(SRC[:-2] + ".h").read())
    lib = oracle.load(oracle.build(str(mut), str(tmp_path / "libmut.so")))
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            pin(lib)
        except AssertionError as exc:
            caught.append(f"{pin.__name__}: {str(exc)[:80]}")
            break
    assert caught, f"mutant {name} passed every pin"
