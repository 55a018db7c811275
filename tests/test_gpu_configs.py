"""Each benchmark workload at the staging its configuration states, compared element by
element with the oracle: the whole layout, every packed row (on the device and, with host
staging, in the pinned bounce buffer the SDMA leg filled), and every combined token.

  tiny    T=128,  H=1024, 16 experts top-2, R=4:   HBM staging
  coarse  T=4096, H=4096, 8 experts top-2,  R=4:   HBM and pinned-host staging
  fine    T=8192, H=2048, 128 experts top-8, R=8:  pinned-host staging through SDMA (the
          default legs and the per-sender mode)
  decode  T=256,  H=7168, 256 experts top-8, R=8:  pinned-host staging with host flags:
          the one-kernel dispatch and its SDMA leg, then the combine after the simulated
          peers, which wait for this rank's flags before raising theirs, over rounds on
          alternating buffer sets
The 32768-token prefill layer is in test_gpu_fullsize.py.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import compare_combine, compare_packed_rows, say
from paper_2609_40093_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
LAYOUT_KEYS = ("expert_counts", "expert_offsets", "rank_counts", "rank_offsets", "slot_pos", "row_src")


@pytest.fixture(scope="module", autouse=True)
def oracle_on_all_cores():
    oracle.set_threads(len(os.sched_getaffinity(0)))
    yield
    oracle.set_threads(1)


def inputs(name):
    cfg = synth.config(name)
    inp = synth.make_inputs(cfg)
    ref = oracle.layout(inp.topk_idx, cfg.E, cfg.R)
    assert ref.status == oracle.OK
    return cfg, inp, inp.expert_outputs(), ref


def check_round(cfg, inp, y, ref, lay, st, out, buf, what):
    """The layout, every packed row on the device (and in the host bounce buffer with
    pinned staging), and every combined token of one round."""
    n, k = cfg.slots, cfg.k
    for key in LAYOUT_KEYS:
        assert np.array_equal(getattr(lay, key).cpu().numpy(), getattr(ref, key)), f"{what}: {key}"

    def dev_rows(r0, r1):
        return st.read_device("send", r1, buf=buf)[r0:r1].cpu().numpy().view(np.uint16)
    compare_packed_rows(dev_rows, inp.x, ref.row_src, k, n, f"{what}: device send rows")
    if st.kind == "pinned":
        host = st.host_array("send", buf)
        compare_packed_rows(lambda r0, r1: host[r0:r1], inp.x, ref.row_src, k, n, f"{what}: host bounce rows")
    o16 = out.view(torch.int16)
    compare_combine(lambda t0, t1: o16[t0:t1].cpu().numpy().view(np.uint16), y, ref.slot_pos, inp.topk_w,
                    f"{what}: combine")


def run(name, staging, mode=0, rounds=1, expect_one_kernel=None):
    cfg, inp, y, ref = inputs(name)
    T, H, E, k, R, n = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R, cfg.slots
    nbuf = 2 if rounds > 1 else 1
    what = f"{name}, {staging} staging" + (f", mode {mode}" if mode else "")
    say(f"{what}: {rounds} round(s)")
    x = torch.from_numpy(inp.x.view(np.int16)).to(DEV)
    idx = torch.from_numpy(inp.topk_idx).to(DEV)
    w = torch.from_numpy(inp.topk_w).to(DEV)
    st = ep.Staging(staging, n, H, R, num_buffers=nbuf, chunk_bytes=16 << 20)
    peers = None
    if staging == "pinned":
        if mode:
            st.set_mode(mode, self_rank=0)
        for b in range(nbuf):
            st.host_array("recv", b)[:n] = y
        peers = ep.SimPeers(st, echo=False)
    else:
        for b in range(nbuf):
            st.write_device("recv", torch.from_numpy(y.view(np.int16)).to(DEV), buf=b)
    lays = [None] * nbuf
    outs = [torch.empty((T, H), dtype=torch.bfloat16, device=DEV) for _ in range(nbuf)]
    ep.trace_reset()
    ep.trace_enable(True)
    try:
        for r in range(rounds):
            b, epoch = r % nbuf, r + 1
            if peers is not None:
                peers.post(b, epoch, n)   # the peers answer once this round's send flags are up
            lays[b] = ep.dispatch_fused(x, idx, E, R, st, buf=b, epoch=epoch, out=lays[b])
            ep.combine(st, lays[b].slot_pos, w, out=outs[b], buf=b, epoch=epoch, rank_offsets=lays[b].rank_offsets)
            if staging == "pinned":
                st.status()
                flags = st.host_array("send_flags", b)
                used = -(-n * st.row_bytes // st.chunk_bytes)
                assert (flags[:used] == epoch).all(), f"{what}: send flags of round {r}"
                assert (st.host_array("recv_flags", b) == epoch).all(), f"{what}: peers' flags of round {r}"
            torch.cuda.synchronize()
            ep.layout_validate(lays[b])
            check_round(cfg, inp, y, ref, lays[b], st, outs[b], b, f"{what}, round {r}")
    finally:
        ep.trace_enable(False)
        if peers is not None:
            peers.drain()
            peers.close()
    ran = ep.trace_read()
    ep.trace_reset()
    if expect_one_kernel is not None:
        assert ("layout_pack" in ran) == expect_one_kernel, sorted(ran)
    st.close()


def test_tiny_hbm():
    run("tiny", "hbm", expect_one_kernel=True)


@pytest.mark.parametrize("staging", ["hbm", "pinned"])
def test_coarse(staging):
    run("coarse", staging, rounds=2 if staging == "pinned" else 1, expect_one_kernel=True)


@pytest.mark.parametrize("mode", [0, ep.MODE_PER_SENDER])
def test_fine_pinned(mode):
    run("fine", "pinned", mode=mode, rounds=2)


def test_decode_pinned_with_host_flags():
    run("decode", "pinned", rounds=3, expect_one_kernel=True)
