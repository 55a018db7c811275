"""ep_dispatch_layout_static (no workspace argument: the layout's scratch is the library's
own array) against ep_dispatch_layout on the same inputs, through the C ABI: every output
equal bit for bit, and the status word equal to what ep_layout_validate reports, over
calls in a row on one GPU -- the prefill layer's routing (several tiles), then a smaller
one (one tile), then a mid-sized one with other sizes, then one with a repeated expert --
and the first of them checked against the oracle too."""
import numpy as np
import pytest
import torch

import oracle
from gpu_cases import make_case, say
from paper_2609_40093_amd import _lib, api, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
KEYS = ("expert_counts", "expert_offsets", "rank_counts", "rank_offsets", "slot_pos", "row_src")


def layouts(idx: np.ndarray, E: int, R: int):
    """(outputs of ep_dispatch_layout, its validate status, outputs of ep_dispatch_layout_static,
    its status word), every output array pre-filled with a value no layout writes."""
    T, k = idx.shape
    n = max(T * k, 1)
    lib = api._lib_handle()
    i32 = dict(dtype=torch.int32, device=DEV)

    def outs():
        return [torch.full((E,), -7, **i32), torch.full((E + 1,), -7, **i32), torch.full((R,), -7, **i32),
                torch.full((R + 1,), -7, **i32), torch.full((n,), -7, **i32), torch.full((n,), -7, **i32)]
    ref, got = outs(), outs()
    idx_d = torch.from_numpy(np.ascontiguousarray(idx)).to(DEV)
    ws = torch.zeros(api.workspace_bytes(T, k, E), dtype=torch.uint8, device=DEV)
    status = torch.full((1,), 0x7FFF, dtype=torch.int32, device=DEV)
    s = api._stream_ptr(None)
    assert lib.ep_dispatch_layout(api._ptr(idx_d), T, k, E, R, *[api._ptr(t) for t in ref], api._ptr(ws), ws.numel(),
                                  s) == 0, lib.ep_last_error()
    assert lib.ep_dispatch_layout_static(api._ptr(idx_d), T, k, E, R, *[api._ptr(t) for t in got],
                                         api._ptr(status), s) == 0, lib.ep_last_error()
    torch.cuda.synchronize()
    ref_status = lib.ep_layout_validate(api._ptr(ws), s)
    ref = {key: t.cpu().numpy()[:T * k] if key in ("slot_pos", "row_src") else t.cpu().numpy()
           for key, t in zip(KEYS, ref)}
    got = {key: t.cpu().numpy()[:T * k] if key in ("slot_pos", "row_src") else t.cpu().numpy()
           for key, t in zip(KEYS, got)}
    return ref, ref_status, got, int(status.item())


def check_equal(idx, E, R, what, oracle_too=False):
    say(f"static-scratch layout: {what} (T={idx.shape[0]}, k={idx.shape[1]}, E={E}, R={R})")
    ref, ref_status, got, status = layouts(idx, E, R)
    assert ref_status == 0 and status == 0, (ref_status, status)
    for key in KEYS:
        assert np.array_equal(got[key], ref[key]), f"{what}: {key}"
    if oracle_too:
        want = oracle.layout(idx, E, R)
        for key in KEYS:
            assert np.array_equal(got[key], getattr(want, key)), f"{what}: {key} vs the oracle"


def test_static_scratch_layout_matches_the_workspace_layout():
    cfg = synth.config("prefill")
    inp = synth.make_inputs(cfg)
    check_equal(inp.topk_idx, cfg.E, cfg.R, "prefill routing, several tiles", oracle_too=True)
    small = make_case("static_small", 128, 8, 16, 2, 4, "random", seed=3)
    check_equal(small.topk_idx, 16, 4, "smaller routing, one tile")
    mid = make_case("static_mid", 5000, 8, 64, 4, 8, "skewed", seed=4)
    check_equal(mid.topk_idx, 64, 8, "mid-sized routing, other sizes")
    # a repeated expert: the status word carries the same routing error as the workspace's
    bad = mid.topk_idx.copy()
    bad[17, 1] = bad[17, 0]
    say("static-scratch layout: repeated expert")
    _, ref_status, _, status = layouts(bad, 64, 8)
    assert ref_status == _lib.EP_ERR_BAD_ROUTING
    assert status == 2, status   # kRoutingDuplicate
    check_equal(small.topk_idx, 16, 4, "the smaller routing again")
