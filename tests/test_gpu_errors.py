"""Error paths through the C ABI on the GPU: bad routing is reported (never a stray
write), host-checkable mistakes are rejected before anything is enqueued."""
import numpy as np
import pytest
import torch

import paper_2609_40093_amd as ep
from gpu_cases import make_case, say

pytestmark = pytest.mark.gpu

DEV = "cuda"


def test_out_of_range_ids_are_reported():
    say("out-of-range expert ids")
    case = make_case("bad_ids", 5000, 64, 16, 2, 4, "random", seed=1)
    idx = case.topk_idx.copy()
    idx[17, 1] = 16
    idx[4321, 0] = -3
    lay = ep.dispatch_layout(torch.from_numpy(idx).to(DEV), 16, 4)
    with pytest.raises(ep.EPError) as ei:
        ep.layout_status(lay)
    assert ei.value.status == 2 and "outside" in str(ei.value)
    sp = lay.slot_pos.cpu().numpy()
    assert sp[17 * 2 + 1] == -1 and sp[4321 * 2] == -1
    valid = np.delete(sp, [35, 8642])
    assert sorted(valid.tolist()) == list(range(valid.size))       # the rest still a permutation
    # a dispatch with those positions skips the two slots instead of writing out of bounds
    st = ep.Staging("hbm", case.slots, 64, 4, num_buffers=1)
    ep.dispatch(torch.from_numpy(case.x.view(np.int16)).to(DEV), lay.slot_pos, st, topk=2)
    torch.cuda.synchronize()
    st.close()


def test_duplicate_expert_in_a_row_is_reported():
    say("duplicate expert within a token row")
    case = make_case("dup", 300, 64, 16, 4, 4, "random", seed=2)
    idx = case.topk_idx.copy()
    idx[100, 3] = idx[100, 0]
    lay = ep.dispatch_layout(torch.from_numpy(idx).to(DEV), 16, 4)
    with pytest.raises(ep.EPError) as ei:
        ep.layout_status(lay)
    assert ei.value.status == 2 and "repeated" in str(ei.value)
    # the next good routing on the same workspace clears the status
    lay = ep.dispatch_layout(torch.from_numpy(case.topk_idx).to(DEV), 16, 4, out=lay)
    ep.layout_status(lay)


def test_host_checked_arguments():
    say("host-side argument checks")
    case = make_case("args", 64, 256, 16, 2, 4, "random", seed=3)
    lay = ep.dispatch_layout(torch.from_numpy(case.topk_idx).to(DEV), 16, 4)
    x = torch.from_numpy(case.x.view(np.int16)).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    small = ep.Staging("hbm", case.slots - 1, 256, 4, num_buffers=1)
    with pytest.raises(ep.EPError, match="exceed"):
        ep.dispatch(x, lay.slot_pos, small, topk=2)
    other_h = ep.Staging("hbm", case.slots, 128, 4, num_buffers=1)
    with pytest.raises(ep.EPError, match="hidden"):
        ep.dispatch(x, lay.slot_pos, other_h, topk=2)
    st = ep.Staging("hbm", case.slots, 256, 4, num_buffers=2)
    with pytest.raises(ep.EPError, match="buffer"):
        ep.dispatch(x, lay.slot_pos, st, topk=2, buf=2)
    flat = torch.zeros(64 * 256 + 8, dtype=torch.int16, device=DEV)
    misaligned = flat[1:1 + 64 * 256].view(64, 256)
    with pytest.raises(ep.EPError, match="aligned"):
        ep.dispatch(misaligned, lay.slot_pos, st, topk=2)
    out_flat = torch.zeros(64 * 256 + 8, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(ep.EPError, match="aligned"):
        ep.combine(st, lay.slot_pos, w, out=out_flat[1:1 + 64 * 256].view(64, 256))
    for s in (small, other_h, st):
        s.close()


def test_impossible_device_staging_is_oom():
    say("device staging larger than HBM")
    with pytest.raises(ep.EPError) as ei:
        ep.Staging("hbm", 1 << 36, 8192, 8, num_buffers=1)     # 1 PiB per buffer
    assert ei.value.status == 4
