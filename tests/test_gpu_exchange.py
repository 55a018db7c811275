"""Exchange modes of host staging on the GPU: per-sender gating, full-duplex legs and the
remote-only self segment, through the C ABI with simulated peers.

Identity experts and dyadic gates make combine(dispatch(x)) == x exactly, in fp32 and
bf16, whatever path each segment took; every leg's bytes are compared with what it must
carry (the oracle's packed rows, the harness's inbound rows), and the flags with the
epoch.  The per-sender test watches the landed flags on the host while one sender is
held back: the other senders' rows arrive first only under the per-sender policy.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import make_case, say
from paper_2609_40093_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"
PS, DUP, RO = ep.MODE_PER_SENDER, ep.MODE_DUPLEX, ep.MODE_REMOTE_ONLY
SENTINEL = 0xFFFF


def bits(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV)


def wait_host(pred, timeout_s=10.0):
    t0 = time.monotonic()
    while not pred():
        if time.monotonic() - t0 > timeout_s:
            return False
        time.sleep(0.0005)
    return True


MODES = [PS, DUP, DUP | PS, DUP | RO, DUP | RO | PS]


@pytest.mark.parametrize("mode", MODES, ids=["per_sender", "duplex", "duplex_per_sender", "duplex_remote_only",
                                             "duplex_remote_only_per_sender"])
def test_exchange_roundtrip_exact(mode):
    R = 8
    roundtrip(3000, 1024, 64, 4, R, 2, mode, case_seed=21, rng_seed=5, chunk_bytes=1 << 20,
              inbound_us=[(r * 7919) % 3000 for r in range(R)], return_us=[(r * 104729) % 5000 for r in range(R)])


@pytest.mark.parametrize("seed", range(12))
def test_exchange_roundtrip_random_shapes(seed):
    """Seeded random groups (2 to 16 ranks, any self rank), routings, row lengths, chunk
    sizes and modes, with senders answering at once or staggered (so that inbound copies
    of neighbouring senders merge, with their landed flags, or go one by one): the same
    checks as above."""
    rng = np.random.default_rng(1000 + seed)
    R = int(rng.choice([2, 4, 8, 16]))
    E = R * int(rng.choice([1, 2, 8]))
    k = int(rng.choice([kk for kk in (1, 2, 4, 8) if kk <= E]))  # 1/k gates: exact sums
    T = int(rng.integers(1, 2000))
    H = int(rng.choice([512, 1024, 2048]))
    me = int(rng.integers(0, R))
    mode = MODES[int(rng.integers(0, len(MODES)))]
    stagger = bool(rng.integers(0, 2))
    inbound_us = [int(rng.integers(0, 3000)) if stagger else 0 for _ in range(R)]
    return_us = [int(rng.integers(0, 3000)) if stagger else 0 for _ in range(R)]
    chunk = int(rng.choice([64 << 10, 1 << 20]))
    say(f"exchange random case {seed}: T={T} H={H} E={E} k={k} R={R} me={me} mode={mode} stagger={stagger}")
    roundtrip(T, H, E, k, R, me, mode, case_seed=2000 + seed, rng_seed=seed, chunk_bytes=chunk,
              inbound_us=inbound_us, return_us=return_us)


def roundtrip(T, H, E, k, R, me, mode, case_seed, rng_seed, chunk_bytes, inbound_us, return_us):
    """Three rounds on alternating buffer sets with identity experts: combine(dispatch(x))
    == x exactly (fp32), every leg's bytes, the offsets and every flag checked."""
    case = make_case("exchange", T, H, E, k, R, "skewed", seed=case_seed, gates="uniform")
    rows = T * k
    lay_o = oracle.layout(case.topk_idx, E, R)
    ro = lay_o.rank_offsets
    st = ep.Staging("pinned", rows, H, R, num_buffers=2, chunk_bytes=chunk_bytes)
    st.set_mode(mode, self_rank=me)
    peers = ep.SimPeers(st, echo=True)
    peers.set_delays(inbound_us=inbound_us, return_us=return_us)
    rng = np.random.default_rng(rng_seed)
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    lay = ep.dispatch_layout(idx, E, R)
    for rnd in range(3):
        buf, epoch = rnd % 2, 100 + rnd
        say(f"exchange mode {mode} round {rnd}")
        # fresh payload every round (low mantissa bits flipped): stale bytes cannot pass
        xr = case.x ^ np.uint16(rnd + 1)
        x = bits(xr)
        packed = oracle.pack(xr, lay_o.slot_pos, k)
        inbound = None
        if mode & DUP:
            # inbound rows of every sender, all of them within the staging's rows
            cap = max(0, (rows - int(ro[me + 1] - ro[me])) // max(1, R - 1))
            rin = [int(rng.integers(0, min(900, cap) + 1)) for _ in range(R)]
            if rnd == 1:
                rin[(me + 1) % R] = 0   # a sender with no rows for this rank
            rin[me] = 0
            st.set_inbound(buf, rin)
            full = list(rin)
            full[me] = int(ro[me + 1] - ro[me])
            off = np.concatenate([[0], np.cumsum(full)]).astype(np.int64)
            inbound = rng.integers(0, 1 << 16, size=(int(off[-1]), H), dtype=np.uint16)
            st.host_array("in", buf)[:off[-1]] = inbound
            st.host_array("ret", buf)[:] = SENTINEL
        st.host_array("send", buf)[:] = SENTINEL
        peers.post(buf, epoch, rows)
        ep.dispatch(x, lay.slot_pos, st, topk=k, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)
        # identity experts: the rows in dev_in are their own results
        out32 = ep.combine(st, lay.slot_pos, w, out_dtype=torch.float32, buf=buf, epoch=epoch,
                           rank_offsets=lay.rank_offsets)
        st.status()
        peers.drain()
        xf = torch.from_numpy(xr.view(np.int16)).view(torch.bfloat16).float()
        assert torch.equal(out32.cpu(), xf), "combine(dispatch(x)) != x"
        hs = st.host_array("send", buf)[:rows]
        for r in range(R):
            seg = slice(int(ro[r]), int(ro[r + 1]))
            if r == me and mode & RO:
                assert np.all(hs[seg] == SENTINEL), "own segment crossed PCIe in remote-only mode"
            else:
                assert np.array_equal(hs[seg], packed[seg]), f"host send segment {r} differs"
        sf = st.host_array("send_flags", buf)
        nchunks = (rows * 2 * H + st.chunk_bytes - 1) // st.chunk_bytes
        assert np.all(sf[:nchunks] == epoch)
        if mode & DUP:
            din = st.read_device("in", int(off[-1]), buf).cpu().numpy().view(np.uint16)
            inl, retf = st.host_array("in_landed", buf), st.host_array("ret_flags", buf)
            hret = st.host_array("ret", buf)
            assert np.array_equal(st.host_array("in_offsets", buf), off)
            for r in range(R):
                seg = slice(int(off[r]), int(off[r + 1]))
                want = packed[int(ro[me]):int(ro[me + 1])] if r == me else inbound[seg]
                assert np.array_equal(din[seg], want), f"inbound rows of sender {r} differ"
                if r == me and mode & RO:
                    assert np.all(hret[seg] == SENTINEL)
                    continue
                assert np.array_equal(hret[seg], din[seg]), f"outbound results for rank {r} differ"
                if off[r + 1] > off[r]:
                    assert inl[r] == epoch and retf[r] == epoch
        rl = st.host_array("recv_landed", buf)
        for r in range(R):
            if ro[r + 1] > ro[r] and not (r == me and mode & RO):
                assert rl[r] == epoch, f"recv_landed[{r}] = {rl[r]}"
    peers.close()
    st.close()


@pytest.mark.parametrize("per_sender", [True, False], ids=["per_sender", "all_senders"])
def test_ready_senders_land_before_a_late_one(per_sender):
    """Sender 1 is held back 1 s: with the per-sender policy every other sender's rows
    land meanwhile; with the all-senders policy none does."""
    T, H, E, k, R = 2048, 2048, 32, 2, 4
    case = make_case("late_sender", T, H, E, k, R, "random", seed=22, gates="uniform")
    rows = T * k
    st = ep.Staging("pinned", rows, H, R, num_buffers=1)
    if per_sender:
        st.set_mode(PS)
    else:
        # the exchange engine's all-senders policy: duplex legs with no inbound rows
        st.set_mode(DUP)
        st.set_inbound(0, [0] * R)
    peers = ep.SimPeers(st, echo=True)
    peers.set_delays(return_us=[0, 1_000_000, 0, 0])
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    lay = ep.dispatch_layout(idx, E, R)
    ro = lay.rank_offsets.cpu().numpy()
    w = torch.from_numpy(case.topk_w).to(DEV)
    epoch = 7
    say(f"late sender, per_sender={per_sender}")
    t0 = time.monotonic()
    peers.post(0, epoch, rows)
    ep.dispatch(bits(case.x), lay.slot_pos, st, topk=k, epoch=epoch, rank_offsets=lay.rank_offsets)
    out = ep.combine(st, lay.slot_pos, w, out_dtype=torch.float32, epoch=epoch, rank_offsets=lay.rank_offsets)
    rl = st.host_array("recv_landed")
    others = [r for r in (2, 3) if ro[r + 1] > ro[r]]
    assert others, "routing left senders 2 and 3 empty"
    if per_sender:
        assert wait_host(lambda: all(rl[r] == epoch for r in others), 5.0), "ready senders never landed"
        assert rl[1] != epoch and time.monotonic() - t0 < 1.0, "late sender landed too early"
    else:
        time.sleep(0.15)
        assert all(rl[r] != epoch for r in others), "all-senders policy started before the last flag"
    st.status()
    peers.drain()
    xf = torch.from_numpy(case.x.view(np.int16)).view(torch.bfloat16).float()
    assert torch.equal(out.cpu(), xf)
    peers.close()
    st.close()


ACC = ep.MODE_ACCUMULATE
# return delays of the 8 senders (us after the round is posted)
ARRIVALS = {
    "at_once": [0] * 8,
    "first_late": [250_000] + [0] * 7,
    "last_late": [0] * 7 + [250_000],
    "reversed": [(8 - r) * 30_000 for r in range(8)],
    "staggered": [(r * 104729) % 150_000 for r in range(8)],
}


@pytest.mark.parametrize("arrival", sorted(ARRIVALS))
@pytest.mark.parametrize("mode", [PS | ACC, DUP | PS | ACC, DUP | RO | PS | ACC],
                         ids=["per_sender_acc", "duplex_per_sender_acc", "duplex_remote_only_per_sender_acc"])
def test_accumulate_equals_single_reduction(mode, arrival):
    """EP_MODE_ACCUMULATE reduces each sender's rows as they land, yet every token's rows
    go in slot order: the output equals the single reduction of the same landed rows bit
    for bit (bf16 and fp32), whatever the arrival order, and the oracle within tolerance."""
    T, H, E, k, R, me = 1000, 512, 64, 8, 8, 3
    case = make_case("accumulate", T, H, E, k, R, "skewed", seed=23)
    rows = T * k
    lay_o = oracle.layout(case.topk_idx, E, R)
    ro = lay_o.rank_offsets
    st = ep.Staging("pinned", rows, H, R, num_buffers=2, chunk_bytes=1 << 20)
    st.set_mode(mode, self_rank=me)
    peers = ep.SimPeers(st, echo=True)
    peers.set_delays(inbound_us=[0] * R, return_us=ARRIVALS[arrival])
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    lay = ep.dispatch_layout(idx, E, R)
    rng = np.random.default_rng(6)
    for rnd, dt in enumerate((torch.bfloat16, torch.float32)):
        buf, epoch = rnd % 2, 50 + rnd
        say(f"accumulate mode {mode} arrival {arrival} round {rnd}")
        xr = case.x ^ np.uint16(rnd + 1)
        if mode & DUP:
            rin = [int(rng.integers(0, 300)) for _ in range(R)]
            rin[me] = 0
            st.set_inbound(buf, rin)
            n_in = sum(rin) + int(ro[me + 1] - ro[me])
            st.host_array("in", buf)[:n_in] = synth.normal_bf16_rows(np.random.SeedSequence([9, rnd]), n_in, H)
        peers.post(buf, epoch, rows)
        ep.dispatch(bits(xr), lay.slot_pos, st, topk=k, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)
        out = ep.combine(st, lay.slot_pos, w, out_dtype=dt, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)
        st.status()
        peers.drain()
        ref = torch.empty_like(out)
        ep.combine_rows(st.read_device("recv", rows, buf), lay.slot_pos, w, ref)
        iv = torch.int16 if dt == torch.bfloat16 else torch.int32
        assert torch.equal(out.view(iv), ref.view(iv)), "accumulated combine != single reduction"
        exact, _, _ = oracle.combine(oracle.pack(xr, lay_o.slot_pos, k), lay_o.slot_pos, case.topk_w)
        got = out.float().cpu().numpy().astype(np.float64)
        err = np.abs(got - exact)
        assert err.max() <= 2e-2 and err.mean() <= 2e-3
    peers.close()
    st.close()


@pytest.mark.parametrize("seed", range(8))
def test_accumulate_random_shapes(seed):
    """Seeded random groups, routings, row lengths (any multiple of 8 elements), top-k and
    arrival delays through the accumulation as senders land: the output equals the single
    reduction of the same landed rows bit for bit, and the oracle within tolerance."""
    rng = np.random.default_rng(5000 + seed)
    R = int(rng.choice([2, 4, 8, 16]))
    E = R * int(rng.choice([1, 2, 8]))
    k = int(rng.integers(1, min(8, E) + 1))
    T = int(rng.integers(1, 1500))
    H = int(rng.choice([8, 264, 512, 1032, 2048]))
    me = int(rng.integers(0, R))
    mode = [PS | ACC, DUP | PS | ACC, DUP | RO | PS | ACC][int(rng.integers(0, 3))]
    delays = [int(rng.integers(0, 20_000)) for _ in range(R)]
    say(f"accumulate random case {seed}: T={T} H={H} E={E} k={k} R={R} me={me} mode={mode}")
    case = make_case("accumulate_random", T, H, E, k, R, "random", seed=6000 + seed)
    rows = T * k
    lay_o = oracle.layout(case.topk_idx, E, R)
    ro = lay_o.rank_offsets
    st = ep.Staging("pinned", rows, H, R, num_buffers=2, chunk_bytes=1 << 20)
    st.set_mode(mode, self_rank=me)
    peers = ep.SimPeers(st, echo=True)
    peers.set_delays(inbound_us=[0] * R, return_us=delays)
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    lay = ep.dispatch_layout(idx, E, R)
    for rnd in range(2):
        buf, epoch = rnd % 2, 70 + rnd
        xr = case.x ^ np.uint16(rnd + 1)
        if mode & DUP:
            cap = max(0, (rows - int(ro[me + 1] - ro[me])) // max(1, R - 1))
            rin = [int(rng.integers(0, min(300, cap) + 1)) for _ in range(R)]
            rin[me] = 0
            st.set_inbound(buf, rin)
            n_in = sum(rin) + int(ro[me + 1] - ro[me])
            st.host_array("in", buf)[:n_in] = synth.normal_bf16_rows(np.random.SeedSequence([19, seed, rnd]), n_in, H)
        peers.post(buf, epoch, rows)
        ep.dispatch(bits(xr), lay.slot_pos, st, topk=k, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)
        out = ep.combine(st, lay.slot_pos, w, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)
        st.status()
        peers.drain()
        ref = torch.empty_like(out)
        ep.combine_rows(st.read_device("recv", rows, buf), lay.slot_pos, w, ref)
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), "accumulated combine != single reduction"
        exact, _, _ = oracle.combine(oracle.pack(xr, lay_o.slot_pos, k), lay_o.slot_pos, case.topk_w)
        err = np.abs(out.float().cpu().numpy().astype(np.float64) - exact)
        assert err.max() <= 2e-2 and err.mean() <= 2e-3
    peers.close()
    st.close()


def test_accumulate_reduces_before_a_late_sender_lands():
    """Sender 1 is held back 0.6 s.  Meanwhile every token none of whose rows comes from it
    is already final in the output (read from another stream while the combine still waits),
    and every other token is still unwritten."""
    T, H, E, k, R = 2048, 1024, 32, 2, 4
    case = make_case("acc_late", T, H, E, k, R, "random", seed=24)
    rows = T * k
    st = ep.Staging("pinned", rows, H, R, num_buffers=1)
    st.set_mode(PS | ACC)
    peers = ep.SimPeers(st, echo=True)
    peers.set_delays(return_us=[0, 600_000, 0, 0])
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    lay = ep.dispatch_layout(idx, E, R)
    ro = lay.rank_offsets.cpu().numpy()
    w = torch.from_numpy(case.topk_w).to(DEV)
    out = torch.full((T, H), float("nan"), dtype=torch.float32, device=DEV)
    torch.cuda.synchronize()
    epoch = 5
    say("accumulate with a late sender")
    peers.post(0, epoch, rows)
    ep.dispatch(bits(case.x), lay.slot_pos, st, topk=k, epoch=epoch, rank_offsets=lay.rank_offsets)
    ep.combine(st, lay.slot_pos, w, out=out, epoch=epoch, rank_offsets=lay.rank_offsets)
    rl = st.host_array("recv_landed")
    assert wait_host(lambda: all(rl[r] == epoch for r in (0, 2, 3) if ro[r + 1] > ro[r]), 5.0)
    time.sleep(0.1)  # the passes for the ready senders run within milliseconds
    side = torch.cuda.Stream()
    snap = torch.empty((T, H), dtype=torch.float32, pin_memory=True)
    with torch.cuda.stream(side):
        snap.copy_(out, non_blocking=True)
    side.synchronize()
    assert rl[1] != epoch, "the late sender landed before the snapshot"
    st.status()
    peers.drain()
    final = out.cpu()
    sender = np.searchsorted(ro, lay.slot_pos.cpu().numpy(), side="right").reshape(T, k) - 1
    early = torch.from_numpy(~(sender == 1).any(axis=1))
    assert early.any() and (~early).any()
    assert torch.equal(snap[early], final[early]), "tokens of landed senders not final before the late one"
    assert torch.isnan(snap[~early]).all(), "a token waiting for the late sender was written early"
    peers.close()
    st.close()


def test_exchange_argument_errors():
    say("exchange argument errors")
    hbm = ep.Staging("hbm", 64, 64, 4, num_buffers=1)
    with pytest.raises(ep.EPError, match="PINNED_HOST"):
        hbm.set_mode(PS)
    hbm.close()
    st = ep.Staging("pinned", 64, 64, 4, num_buffers=1)
    with pytest.raises(ep.EPError, match="needs EP_MODE_DUPLEX"):
        st.set_mode(RO)
    with pytest.raises(ep.EPError, match="needs EP_MODE_PER_SENDER"):
        st.set_mode(ep.MODE_ACCUMULATE)
    with pytest.raises(ep.EPError, match="self_rank"):
        st.set_mode(PS, self_rank=4)
    with pytest.raises(ep.EPError, match="exceed"):
        st.set_inbound(0, [0, 40, 40, 0])
    big = ep.Staging("pinned", 64, 64, 33, num_buffers=1)
    with pytest.raises(ep.EPError, match="at most 32"):
        big.set_mode(PS)
    big.close()
    st.set_mode(DUP)
    case = make_case("args", 16, 64, 8, 2, 4, "random", seed=3)
    lay = ep.dispatch_layout(torch.from_numpy(case.topk_idx).to(DEV), 8, 4)
    with pytest.raises(ep.EPError, match="rank_offsets"):
        ep.dispatch(bits(case.x), lay.slot_pos, st, topk=2, epoch=3)
    w = torch.from_numpy(case.topk_w).to(DEV)
    with pytest.raises(ep.EPError, match="duplex dispatch"):
        ep.combine(st, lay.slot_pos, w, epoch=9, rank_offsets=lay.rank_offsets)
    torch.cuda.synchronize()
    st.close()


def test_pcie_probe_runs_both_directions():
    say("pcie probe")
    n = 64 << 20
    host = torch.empty(2 * n, dtype=torch.uint8, pin_memory=True)
    dev = torch.empty(2 * n, dtype=torch.uint8, device=DEV)
    rates = [ep.pcie_probe(host, dev, n, d) for d in (1, 2, 3)]
    assert all(r > 1.0 for r in rates), rates
