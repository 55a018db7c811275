"""The oracle's pack and combine split over host threads (the all-cores CPU baseline) give
outputs identical, bit for bit, to the single-threaded oracle: each token's rows and sums
are formed by one thread in the same order."""
import numpy as np
import pytest

import oracle
from paper_2609_40093_amd import synth


@pytest.mark.parametrize("name", ["tiny", "decode"])
def test_threads_do_not_change_the_outputs(name):
    cfg = synth.config(name)
    inp = synth.make_inputs(cfg)
    y = inp.expert_outputs()
    lay = oracle.layout(inp.topk_idx, cfg.E, cfg.R)
    try:
        assert oracle.set_threads(1) == 1
        p1 = oracle.pack(inp.x, lay.slot_pos, cfg.k)
        e1, b1, f1 = oracle.combine(y, lay.slot_pos, inp.topk_w)
        got = oracle.set_threads(7)
        p7 = oracle.pack(inp.x, lay.slot_pos, cfg.k)
        e7, b7, f7 = oracle.combine(y, lay.slot_pos, inp.topk_w)
    finally:
        oracle.set_threads(1)
    assert got == 7
    assert np.array_equal(p1, p7)
    assert np.array_equal(e1.view(np.uint64), e7.view(np.uint64))
    assert np.array_equal(b1, b7)
    assert np.array_equal(f1.view(np.uint32), f7.view(np.uint32))
