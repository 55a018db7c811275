"""The 32768-token prefill layer (H=7168, 256 experts, top-8, 8 ranks) at full size,
with HBM and with pinned-host staging, in the launch configuration bench.py uses.

Every output is compared with the oracle: the whole layout (262144 routing entries),
all 262144 packed rows (3.76 GB, on the device and, with host staging, in the pinned
bounce buffer the SDMA leg filled), copied back and checked in slices, and all 32768
combined tokens, checked against the oracle's sums in slices of 2048 tokens.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import TOL_MAX_ABS, TOL_MEAN_ABS, combine_errors, compare_combine, compare_packed_rows, routing, say
from paper_2609_40093_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def prefill():
    say("prefill: generating inputs (3.8 GB of expert outputs)")
    cfg = synth.config("prefill")
    inp = synth.make_inputs(cfg)
    y = inp.expert_outputs()
    lay = oracle.layout(inp.topk_idx, cfg.E, cfg.R)
    assert lay.status == oracle.OK
    oracle.set_threads(len(os.sched_getaffinity(0)))
    yield cfg, inp, y, lay
    oracle.set_threads(1)


@pytest.mark.parametrize("staging", ["hbm", "pinned"])
def test_prefill_full_size(prefill, staging):
    cfg, inp, y, ref = prefill
    T, H, E, k, R = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R
    n = cfg.slots
    say(f"prefill full size, {staging} staging: layout")
    idx = torch.from_numpy(inp.topk_idx).to(DEV)
    lay = ep.dispatch_layout(idx, E, R)
    ep.layout_validate(lay)
    for key in ("expert_counts", "expert_offsets", "rank_counts", "rank_offsets", "slot_pos", "row_src"):
        assert np.array_equal(getattr(lay, key).cpu().numpy(), getattr(ref, key)), key

    say(f"prefill full size, {staging} staging: dispatch + combine")
    st = ep.Staging(staging, n, H, R, num_buffers=1, chunk_bytes=16 << 20)
    x = torch.from_numpy(inp.x.view(np.int16)).to(DEV)
    w = torch.from_numpy(inp.topk_w).to(DEV)
    if staging == "hbm":
        ep.dispatch(x, lay.slot_pos, st, topk=k, epoch=3)
        st.write_device("recv", torch.from_numpy(y.view(np.int16)).to(DEV))
        out = ep.combine(st, lay.slot_pos, w, epoch=3)
        torch.cuda.synchronize()
    else:
        st.host_array("recv", 0)[:n] = y
        peers = ep.SimPeers(st, echo=False)
        peers.post(0, 3, n)
        ep.dispatch(x, lay.slot_pos, st, topk=k, epoch=3)
        out = ep.combine(st, lay.slot_pos, w, epoch=3)
        st.status()
        peers.drain()
        peers.close()
        used = -(-n * st.row_bytes // st.chunk_bytes)
        flags = st.host_array("send_flags", 0)
        assert (flags[:used] == 3).all()
        say("prefill full size, pinned staging: every host bounce row")
        host = st.host_array("send", 0)
        compare_packed_rows(lambda r0, r1: host[r0:r1], inp.x, ref.row_src, k, n, "host bounce rows")

    say(f"prefill full size, {staging} staging: every packed row on the device")
    send = st.read_device("send", n)
    torch.cuda.synchronize()
    compare_packed_rows(lambda r0, r1: send[r0:r1].cpu().numpy().view(np.uint16), inp.x, ref.row_src, k, n,
                        "device packed rows")
    del send
    say(f"prefill full size, {staging} staging: every combined token")
    o16 = out.view(torch.int16)
    compare_combine(lambda t0, t1: o16[t0:t1].cpu().numpy().view(np.uint16), y, ref.slot_pos, inp.topk_w,
                    "combine")
    st.close()


def test_coarse_layer_as_the_benchmark_runs_it():
    """The layer the benchmark's value is measured on (T=4096, H=4096, 8 experts, top-2, 4
    ranks, HBM staging), in its launch configuration: one-kernel dispatch then combine,
    over 5 rotated buffer sets, each with its own copies of the inputs, for 3 rounds of the
    sets with layout objects and outputs reused.  Afterwards every set holds the oracle's
    layout and packed rows bit for bit and a combine within tolerance."""
    say("coarse layer, benchmark launch configuration")
    cfg = synth.config("coarse")
    inp = synth.make_inputs(cfg)
    y = inp.expert_outputs()
    T, H, E, k, R = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R
    n, nsets = cfg.slots, 5
    ref = oracle.layout(inp.topk_idx, E, R)
    packed_ref = oracle.pack(inp.x, ref.slot_pos, k)
    exact, _, _ = oracle.combine(y, ref.slot_pos, inp.topk_w)
    x_d = torch.from_numpy(inp.x.view(np.int16)).to(DEV)
    idx_d = torch.from_numpy(inp.topk_idx).to(DEV)
    w_d = torch.from_numpy(inp.topk_w).to(DEV)
    y_d = torch.from_numpy(y.view(np.int16)).to(DEV)
    st = ep.Staging("hbm", n, H, R, num_buffers=nsets)
    sets = []
    for s in range(nsets):
        sets.append(dict(x=x_d.clone(), idx=idx_d.clone(), w=w_d.clone(), lay=None,
                         out=torch.empty((T, H), dtype=torch.bfloat16, device=DEV)))
        st.write_device("recv", y_d, buf=s)
    ep.trace_reset()
    ep.trace_enable(True)
    for i in range(3 * nsets):
        s = sets[i % nsets]
        s["lay"] = ep.dispatch_fused(s["x"], s["idx"], E, R, st, buf=i % nsets, epoch=i + 1, out=s["lay"])
        ep.combine(st, s["lay"].slot_pos, s["w"], out=s["out"], buf=i % nsets, epoch=i + 1)
    torch.cuda.synchronize()
    ep.trace_enable(False)
    assert "layout_pack" in ep.trace_read(), "the one-kernel dispatch did not run"
    ep.trace_reset()
    for b, s in enumerate(sets):
        ep.layout_validate(s["lay"])
        for key in ("expert_counts", "expert_offsets", "rank_counts", "rank_offsets", "slot_pos", "row_src"):
            assert np.array_equal(getattr(s["lay"], key).cpu().numpy(), getattr(ref, key)), f"set {b}: {key}"
        packed = st.read_device("send", n, buf=b).cpu().numpy().view(np.uint16)
        assert packed.tobytes() == packed_ref.tobytes(), f"set {b}: packed rows"
        mx, mean = combine_errors(s["out"].view(torch.int16).cpu().numpy().view(np.uint16), exact)
        assert mx <= TOL_MAX_ABS and mean <= TOL_MEAN_ABS, f"set {b}: combine max {mx} mean {mean}"
    st.close()


@pytest.mark.parametrize("k,H,T", [(8, 7176, 18720), (16, 7168, 9400), (4, 4096, 65600), (2, 7168, 74900),
                                   (2, 7176, 74820)])
def test_write_through_pack_instances(k, H, T):
    """Pack launches that write 2 GiB or more use the write-through store instances: the
    per-slot kernel with rows that are not whole 64-vector groups (H = 7176), with 16-wave
    workgroups (k = 16) and with 4-wave ones (k = 4), and the one-wave-per-chunk kernel
    (k = 2) with whole-group and with ragged rows.  Every packed row is compared with the
    pack definition."""
    E, R = 64, 8
    n = T * k
    assert n * 2 * H >= 2 << 30, "the case must write at least 2 GiB"
    say(f"write-through pack instance: T={T} H={H} k={k}")
    idx = routing("random", T, E, k, seed=T)
    ref = oracle.layout(idx, E, R)
    assert ref.status == oracle.OK
    x = synth.normal_bf16_rows(np.random.SeedSequence([11, T, H, k]), T, H)
    x_d = torch.from_numpy(x.view(np.int16)).to(DEV)
    sp_d = torch.from_numpy(ref.slot_pos).to(DEV)
    out = torch.empty((n, H), dtype=torch.int16, device=DEV)
    ep.pack(x_d, sp_d, out, topk=k)
    torch.cuda.synchronize()
    del x_d
    compare_packed_rows(lambda r0, r1: out[r0:r1].cpu().numpy().view(np.uint16), x, ref.row_src, k, n,
                        f"write-through pack T={T} H={H} k={k}")
