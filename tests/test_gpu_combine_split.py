"""A combine whose output reaches 128 MiB runs as several launches over consecutive token
ranges; below that it is one launch.  Each token's sum is the same arithmetic either way,
so the output of one call over T tokens must equal, bit for bit, the outputs of calls over
slices of the tokens (each slice small enough for one launch), and lie within the
tolerance of the oracle's exact sums.  Cases: bf16 output just past the split size with a
ragged last range, and fp32 output past it (rows twice as long); top-2 keeps the
returned rows to a few hundred MiB.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import TOL_MAX_ABS, compare_combine, make_case, say

pytestmark = pytest.mark.gpu
DEV = "cuda"
SPLIT = 128 << 20


def run(case, out_dtype):
    lay = oracle.layout(case.topk_idx, case.E, case.R)
    assert lay.status == oracle.OK
    st = ep.Staging("hbm", case.slots, case.H, case.R, num_buffers=1)
    st.write_device("recv", torch.from_numpy(case.y.view(np.int16)).to(DEV))
    sp = torch.from_numpy(lay.slot_pos).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    T, k = case.T, case.k
    whole = ep.combine(st, sp, w, out_dtype=out_dtype)
    # the same tokens in slices, each one launch
    slices = torch.empty_like(whole)
    step = -(-T // 5)
    for t0 in range(0, T, step):
        t1 = min(T, t0 + step)
        ep.combine(st, sp[t0 * k:t1 * k], w[t0:t1], out=slices[t0:t1])
    torch.cuda.synchronize()
    st.close()
    return lay, whole, slices


@pytest.mark.parametrize("T,H,out_dtype", [(32771, 2048, torch.bfloat16), (16385, 2048, torch.float32)],
                         ids=["bf16_past_the_split", "fp32_past_the_split"])
def test_split_combine_equals_sliced_calls_and_the_oracle(T, H, out_dtype):
    k, E, R = 2, 16, 4
    row_bytes = H * (2 if out_dtype == torch.bfloat16 else 4)
    assert T * row_bytes >= SPLIT and (-(-T // 5)) * row_bytes < SPLIT
    case = make_case("combine_split", T, H, E, k, R, "random", seed=51)
    say(f"combine over {T} tokens in token-range launches ({out_dtype}), against sliced calls and the oracle")
    lay, whole, slices = run(case, out_dtype)
    a = whole.view(torch.int16 if out_dtype == torch.bfloat16 else torch.int32).cpu().numpy()
    b = slices.view(torch.int16 if out_dtype == torch.bfloat16 else torch.int32).cpu().numpy()
    assert np.array_equal(a, b), f"{int((a != b).any(axis=1).sum())} tokens differ from the sliced calls"
    if out_dtype == torch.bfloat16:
        compare_combine(lambda t0, t1: a[t0:t1].view(np.uint16), case.y, lay.slot_pos, case.topk_w,
                        "split combine")
    else:
        got = whole.cpu().numpy().astype(np.float64)
        for t0 in range(0, T, 4096):
            t1 = min(T, t0 + 4096)
            exact, _, _ = oracle.combine_tokens(case.y[lay.slot_pos[t0 * k:t1 * k]], case.topk_w[t0:t1])
            err = np.abs(got[t0:t1] - exact)
            assert float(err.max()) <= TOL_MAX_ABS, f"fp32 split combine error {float(err.max())} in [{t0}, {t1})"
