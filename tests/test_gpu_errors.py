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
        ep.layout_validate(lay)
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
        ep.layout_validate(lay)
    assert ei.value.status == 2 and "repeated" in str(ei.value)
    # the next good routing on the same workspace clears the status
    lay = ep.dispatch_layout(torch.from_numpy(case.topk_idx).to(DEV), 16, 4, out=lay)
    ep.layout_validate(lay)


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


def test_binding_rejects_host_and_misshaped_tensors():
    """The binding refuses, before any library call, tensors the kernels or engines would
    read as device (or pinned) memory but are not: host tensors, strided views, the wrong
    block dtype, and row counts beyond a staging buffer."""
    say("binding argument checks")
    N, H, k, R = 16, 64, 2, 4
    slot_pos = torch.zeros(N * k, dtype=torch.int32, device=DEV)
    w = torch.full((N, k), 0.5, dtype=torch.float32, device=DEV)
    y = torch.zeros((N * k, H), dtype=torch.int16, device=DEV)
    out = torch.zeros((N, H), dtype=torch.float32, device=DEV)
    with pytest.raises(ValueError, match="y must be a device tensor"):
        ep.combine_rows(y.cpu(), slot_pos, w, out)
    with pytest.raises(ValueError, match="out must be a device tensor"):
        ep.combine_rows(y, slot_pos, w, out.cpu())
    with pytest.raises(ValueError, match="out must be contiguous"):
        ep.combine_rows(y, slot_pos, w, torch.zeros((H, N), dtype=torch.float32, device=DEV).t())
    with pytest.raises(ValueError, match="dst must be a device tensor"):
        ep.copy_probe(torch.empty(64, dtype=torch.uint8), torch.empty(64, dtype=torch.uint8, device=DEV))
    with pytest.raises(ValueError, match="pinned"):
        ep.pcie_probe(torch.empty(128, dtype=torch.uint8), torch.empty(128, dtype=torch.uint8, device=DEV), 64, 1)
    st = ep.Staging("pinned", N * k, H, R, num_buffers=1)
    with pytest.raises(ValueError, match="rows must be in"):
        st.read_device("send", N * k + 1)
    with pytest.raises(ValueError, match="out must be a device tensor"):
        ep.combine_graph(st, slot_pos, w, out.cpu())
    st.close()
    d = ep.Dense(N, H, R, self_rank=0, num_buffers=1, block_dtype=torch.float32)
    with pytest.raises(ValueError, match="blocks must be a device tensor"):
        ep.reducescatter(d, torch.zeros((R * N, H), dtype=torch.float32), num_tokens=N)
    with pytest.raises(ValueError, match="blocks has dtype"):
        ep.reducescatter(d, torch.zeros((R * N, H), dtype=torch.int16, device=DEV), num_tokens=N)
    with pytest.raises(ValueError, match="rows must be in"):
        d.device_rows("gathered", R * N + 1)
    d.close()
