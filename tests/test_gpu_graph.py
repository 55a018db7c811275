"""Graph-replayed rounds (decode): a device round counter picks the buffer set, credits
guard its reuse, and the rows move either on the compute units to and from pinned memory
(legs="cu") or on SDMA engines driven by the library's host-leg thread (legs="sdma",
ep_graph_legs_sdma): the captured kernels then pack into and reduce from device memory.

A round = ep_round_advance, layout, ep_dispatch_graph, ep_combine_graph.  Simulated peers
echo the rows (identity experts), so with dyadic gates every round returns x exactly.
The same round is run eagerly and captured once in a HIP graph and replayed; between
replays new rows and a new routing are written into the captured input buffers, so a
replay that reused stale rows, a stale layout, a stale buffer set or a stale round number
fails.
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


LEGS = ["cu", "sdma"]


def setup(T=256, H=1024, E=64, k=8, R=8, delay_us=0, seed=31, legs="cu"):
    case = make_case("graph", T, H, E, k, R, "random", seed=seed, gates="uniform")
    rows = T * k
    st = ep.Staging("pinned", rows, H, R, num_buffers=2)
    peers = ep.SimPeers(st, echo=True, graph_rows=rows, graph_delay_us=delay_us)
    if legs == "sdma":
        ep.graph_legs_sdma(st, True)
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    x = torch.zeros((T, H), dtype=torch.int16, device=DEV)
    out = torch.empty((T, H), dtype=torch.float32, device=DEV)
    lay = ep.dispatch_layout(idx, E, R)
    return case, st, peers, idx, w, x, out, lay


def one_round(st, idx, w, x, out, lay, case):
    ep.round_advance(st)
    ep.dispatch_layout(idx, case.E, case.R, out=lay)
    ep.dispatch_graph(x, lay.slot_pos, st, topk=case.k)
    ep.combine_graph(st, lay.slot_pos, w, out)


def payload(case, r):
    return synth.normal_bf16_rows(np.random.SeedSequence([77, r]), case.T, case.H)


def as_f32(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32)


@pytest.mark.parametrize("legs", LEGS)
def test_graph_rounds_eager(legs):
    case, st, peers, idx, w, x, out, lay = setup(legs=legs)
    packed_slots = oracle.layout(case.topk_idx, case.E, case.R).slot_pos
    for r in range(1, 6):
        say(f"graph round eager {r} ({legs} legs)")
        xr = payload(case, r)
        x.copy_(torch.from_numpy(xr.view(np.int16)))
        one_round(st, idx, w, x, out, lay, case)
        torch.cuda.synchronize()
        peers.wait_round(r)
        st.status()
        assert np.array_equal(out.cpu().numpy(), as_f32(xr)), f"round {r}"
        b = r % 2
        assert st.host_array("send_flags", b)[0] == r
        assert st.host_array("recv_credit", b)[0] == r, "receive buffer not credited"
        assert np.all(st.host_array("send_credits", b) == r), "peers' credits missing"
        sent = st.host_array("send", b)[:case.slots]
        assert np.array_equal(sent, oracle.pack(xr, packed_slots, case.k)), f"pinned send rows of round {r}"
        if legs == "sdma":  # packed in device memory, then copied by the legs' thread
            dev = st.read_device("send", case.slots, buf=b).cpu().numpy().view(np.uint16)
            assert np.array_equal(dev, sent), f"device send rows of round {r}"
    assert ep.round_read(st) == 5
    peers.close()
    st.close()


@pytest.mark.parametrize("legs", LEGS)
@pytest.mark.parametrize("seed", range(6))
def test_graph_rounds_eager_random_shapes(seed, legs):
    """Seeded random layers through the graph-round path (rows of any multiple of 8
    elements, so also the guarded pack and combine instances; 2 to 8 ranks; top-1 to top-8
    with 1/k gates): three eager rounds, each returning x exactly, with the pinned send
    rows equal to the oracle's pack."""
    rng = np.random.default_rng(4000 + seed)
    R = int(rng.choice([2, 4, 8]))
    E = R * int(rng.choice([1, 2, 8]))
    k = int(rng.choice([kk for kk in (1, 2, 4, 8) if kk <= E]))
    T = int(rng.integers(1, 600))
    H = int(rng.choice([8, 520, 1024, 1032, 7168]))
    say(f"graph rounds random case {seed} ({legs} legs): T={T} H={H} E={E} k={k} R={R}")
    case, st, peers, idx, w, x, out, lay = setup(T=T, H=H, E=E, k=k, R=R, seed=100 + seed, legs=legs)
    packed_slots = oracle.layout(case.topk_idx, case.E, case.R).slot_pos
    for r in range(1, 4):
        xr = payload(case, r)
        x.copy_(torch.from_numpy(xr.view(np.int16)))
        one_round(st, idx, w, x, out, lay, case)
        torch.cuda.synchronize()
        peers.wait_round(r)
        st.status()
        assert np.array_equal(out.cpu().numpy(), as_f32(xr)), f"round {r}"
        sent = st.host_array("send", r % 2)[:case.slots]
        assert np.array_equal(sent, oracle.pack(xr, packed_slots, case.k)), f"pinned send rows of round {r}"
    peers.close()
    st.close()


@pytest.mark.parametrize("legs", LEGS)
def test_graph_capture_replay(legs):
    case, st, peers, idx, w, x, out, lay = setup(seed=32, legs=legs)
    # one eager round first (the layout's device state, kernels loaded)
    xr = payload(case, 0)
    x.copy_(torch.from_numpy(xr.view(np.int16)))
    one_round(st, idx, w, x, out, lay, case)
    torch.cuda.synchronize()
    peers.wait_round(1)
    say("graph capture")
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            one_round(st, idx, w, x, out, lay, case)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    assert ep.round_read(st) == 1, "capture must not run the round"
    for rep in range(6):
        say(f"graph replay {rep} ({legs} legs)")
        xr = payload(case, 100 + rep)
        x.copy_(torch.from_numpy(xr.view(np.int16)))
        # a new routing in the captured routing buffer: the captured layout must recompute
        route = make_case("graph_route", case.T, case.H, case.E, case.k, case.R, "random", seed=200 + rep)
        idx.copy_(torch.from_numpy(route.topk_idx))
        g.replay()
        torch.cuda.synchronize()
        peers.wait_round(2 + rep)
        st.status()
        assert np.array_equal(out.cpu().numpy(), as_f32(xr)), f"replay {rep}"
        assert st.host_array("send_flags", (2 + rep) % 2)[0] == 2 + rep
        ref = oracle.layout(route.topk_idx, case.E, case.R)
        assert np.array_equal(lay.slot_pos.cpu().numpy(), ref.slot_pos), f"replay {rep}: stale layout"
        sent = st.host_array("send", (2 + rep) % 2)[:case.slots]
        assert np.array_equal(sent, oracle.pack(xr, ref.slot_pos, case.k)), f"replay {rep}: pinned send rows"
    assert ep.round_read(st) == 7
    peers.close()
    st.close()


@pytest.mark.parametrize("legs", LEGS)
def test_graph_replays_back_to_back_wait_for_credits(legs):
    """Slow peers (3 ms per round): 8 replays queued without synchronization; the credit
    waits keep every buffer set from being overwritten before the peers consumed it."""
    case, st, peers, idx, w, x, out, lay = setup(delay_us=3000, seed=33, legs=legs)
    xr = payload(case, 5)
    x.copy_(torch.from_numpy(xr.view(np.int16)))
    one_round(st, idx, w, x, out, lay, case)
    torch.cuda.synchronize()
    peers.wait_round(1)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            one_round(st, idx, w, x, out, lay, case)
    torch.cuda.current_stream().wait_stream(s)
    say(f"8 replays back to back ({legs} legs)")
    for _ in range(8):
        g.replay()
    torch.cuda.synchronize()
    peers.wait_round(9)
    st.status()
    assert ep.round_read(st) == 9
    assert np.array_equal(out.cpu().numpy(), as_f32(xr))
    for b in (0, 1):
        assert np.all(st.host_array("send_flags", b)[0] == (9 if b == 1 else 8))
    peers.close()
    st.close()


def test_graph_rounds_need_two_pinned_buffers():
    say("graph argument errors")
    st = ep.Staging("pinned", 64, 64, 4, num_buffers=1)
    with pytest.raises(ep.EPError, match="2 buffer sets"):
        ep.round_advance(st)
    st.close()
    hbm = ep.Staging("hbm", 64, 64, 4, num_buffers=2)
    with pytest.raises(ep.EPError, match="PINNED_HOST"):
        ep.round_advance(hbm)
    hbm.close()


def test_graph_legs_switched_between_rounds():
    """The legs' thread starts at the round the device counter reaches next and stops
    between rounds: two rounds on SDMA legs, two on the compute units, two on SDMA again,
    each returning x exactly with the oracle's rows in the pinned send buffer."""
    case, st, peers, idx, w, x, out, lay = setup(seed=34)
    packed_slots = oracle.layout(case.topk_idx, case.E, case.R).slot_pos
    plan = ["sdma", "sdma", "cu", "cu", "sdma", "sdma"]
    for r, legs in enumerate(plan, start=1):
        if legs != (plan[r - 2] if r > 1 else "cu"):
            ep.graph_legs_sdma(st, legs == "sdma")
        say(f"switched legs: round {r} on {legs}")
        xr = payload(case, 300 + r)
        x.copy_(torch.from_numpy(xr.view(np.int16)))
        one_round(st, idx, w, x, out, lay, case)
        torch.cuda.synchronize()
        peers.wait_round(r)
        st.status()
        assert np.array_equal(out.cpu().numpy(), as_f32(xr)), f"round {r} ({legs})"
        sent = st.host_array("send", r % 2)[:case.slots]
        assert np.array_equal(sent, oracle.pack(xr, packed_slots, case.k)), f"pinned send rows of round {r}"
    ep.graph_legs_sdma(st, False)
    peers.close()
    st.close()


def test_graph_legs_report_peers_that_never_answer():
    """No peers: the legs' thread copies the rows out and raises the send flag, then its
    bounded wait for the senders' flags expires (50 ms).  It records that in the status
    block and still lands the round, so the device's own bounded wait ends too; the status
    call reports the timeout and names the wait."""
    case = make_case("graph_nopeers", 64, 512, 16, 2, 4, "random", seed=35, gates="uniform")
    st = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=2)
    st.set_wait(timeout_us=50_000)
    ep.graph_legs_sdma(st, True)
    idx = torch.from_numpy(case.topk_idx).to(DEV)
    w = torch.from_numpy(case.topk_w).to(DEV)
    x = torch.from_numpy(payload(case, 1).view(np.int16)).to(DEV)
    out = torch.empty((case.T, case.H), dtype=torch.float32, device=DEV)
    lay = ep.dispatch_layout(idx, case.E, case.R)
    say("graph legs with no peers: a bounded wait expires")
    one_round(st, idx, w, x, out, lay, case)
    torch.cuda.synchronize()
    time.sleep(0.3)  # both bounded waits (device and thread) have expired and recorded
    with pytest.raises(ep.EPError) as ei:
        st.status()
    msg = str(ei.value)
    assert "host-leg thread" in msg or "wait_graph_landed" in msg, msg
    # the outbound leg ran: the rows are in the pinned send buffer and the flag is up
    assert st.host_array("send_flags", 1)[0] == 1
    ref = oracle.layout(case.topk_idx, case.E, case.R)
    assert np.array_equal(st.host_array("send", 1)[:case.slots], oracle.pack(payload(case, 1), ref.slot_pos, case.k))
    ep.graph_legs_sdma(st, False)
    st.close()


@pytest.mark.parametrize("legs", LEGS)
def test_graph_replay_at_the_decode_layer_shape(legs):
    """The decode layer's shape (T=256, H=7168, 256 experts top-8, R=8: 29 MB each way per
    round) through captured rounds: every replay returns x exactly (identity experts, gates
    1/8, fp32 output) and leaves the oracle's packed rows in the pinned send buffer."""
    case, st, peers, idx, w, x, out, lay = setup(T=256, H=7168, E=256, k=8, R=8, seed=36, legs=legs)
    xr = payload(case, 0)
    x.copy_(torch.from_numpy(xr.view(np.int16)))
    one_round(st, idx, w, x, out, lay, case)
    torch.cuda.synchronize()
    peers.wait_round(1)
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            one_round(st, idx, w, x, out, lay, case)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    slots = oracle.layout(case.topk_idx, case.E, case.R).slot_pos
    for rep in range(4):
        say(f"decode-shape graph replay {rep} ({legs} legs)")
        xr = payload(case, 400 + rep)
        x.copy_(torch.from_numpy(xr.view(np.int16)))
        g.replay()
        torch.cuda.synchronize()
        peers.wait_round(2 + rep)
        st.status()
        assert np.array_equal(out.cpu().numpy(), as_f32(xr)), f"replay {rep}"
        sent = st.host_array("send", (2 + rep) % 2)[:case.slots]
        assert np.array_equal(sent, oracle.pack(xr, slots, case.k)), f"replay {rep}: pinned send rows"
    peers.close()
    st.close()


@pytest.mark.parametrize("legs", LEGS)
def test_graph_replay_with_a_split_combine(legs):
    """A combine whose fp32 output passes 128 MiB runs as token-range launches; in graph
    rounds each of them reads the round's buffer set (pinned memory with compute-unit legs,
    device memory with SDMA legs).  T=4700 tokens of H=7168, top-2 of 16, R=4 (132 MiB
    each way per round): three replays return x exactly."""
    case, st, peers, idx, w, x, out, lay = setup(T=4700, H=7168, E=16, k=2, R=4, seed=37, legs=legs)
    assert case.T * case.H * 4 >= 128 << 20
    xr = payload(case, 0)
    x.copy_(torch.from_numpy(xr.view(np.int16)))
    one_round(st, idx, w, x, out, lay, case)
    torch.cuda.synchronize()
    peers.wait_round(1)
    st.status()
    assert np.array_equal(out.cpu().numpy(), as_f32(xr)), "eager round"
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            one_round(st, idx, w, x, out, lay, case)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for rep in range(3):
        say(f"split-combine graph replay {rep} ({legs} legs)")
        xr = payload(case, 500 + rep)
        x.copy_(torch.from_numpy(xr.view(np.int16)))
        g.replay()
        torch.cuda.synchronize()
        peers.wait_round(2 + rep)
        st.status()
        assert np.array_equal(out.cpu().numpy(), as_f32(xr)), f"replay {rep}"
    peers.close()
    st.close()
