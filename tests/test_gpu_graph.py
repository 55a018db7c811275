"""Graph-replayed rounds (decode): a device round counter picks the buffer set, credits
guard its reuse, and the rows move on the compute units to and from pinned memory.

A round = ep_round_advance, layout, ep_dispatch_graph, ep_combine_graph.  Simulated peers
echo the rows (identity experts), so with dyadic gates every round returns x exactly.
The same round is run eagerly and captured once in a HIP graph and replayed; between
replays new rows and a new routing are written into the captured input buffers, so a
replay that reused stale rows, a stale layout, a stale buffer set or a stale round number
fails.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import make_case, say
from paper_2609_40093_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def setup(T=256, H=1024, E=64, k=8, R=8, delay_us=0, seed=31):
    case = make_case("graph", T, H, E, k, R, "random", seed=seed, gates="uniform")
    rows = T * k
    st = ep.Staging("pinned", rows, H, R, num_buffers=2)
    peers = ep.SimPeers(st, echo=True, graph_rows=rows, graph_delay_us=delay_us)
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


def test_graph_rounds_eager():
    case, st, peers, idx, w, x, out, lay = setup()
    packed_slots = oracle.layout(case.topk_idx, case.E, case.R).slot_pos
    for r in range(1, 6):
        say(f"graph round eager {r}")
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
    assert ep.round_read(st) == 5
    peers.close()
    st.close()


@pytest.mark.parametrize("seed", range(6))
def test_graph_rounds_eager_random_shapes(seed):
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
    say(f"graph rounds random case {seed}: T={T} H={H} E={E} k={k} R={R}")
    case, st, peers, idx, w, x, out, lay = setup(T=T, H=H, E=E, k=k, R=R, seed=100 + seed)
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


def test_graph_capture_replay():
    case, st, peers, idx, w, x, out, lay = setup(seed=32)
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
        say(f"graph replay {rep}")
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


def test_graph_replays_back_to_back_wait_for_credits():
    """Slow peers (3 ms per round): 8 replays queued without synchronization; the credit
    waits keep every buffer set from being overwritten before the peers consumed it."""
    case, st, peers, idx, w, x, out, lay = setup(delay_us=3000, seed=33)
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
    say("8 replays back to back")
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
