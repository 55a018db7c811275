"""The dense design (All-Gather dispatch, Reduce-Scatter combine) on the GPU against the
oracle, through the C ABI with simulated peer ranks.

  * window layout (grouping the gathered tokens by this rank's experts): bit-exact;
  * pack of the gathered rows into local-expert order: bit-exact;
  * partial blocks (combine over local experts): within the combine tolerance, and exact
    with dyadic gates on small-integer rows;
  * a whole layer -- All-Gather, grouping, identity experts, partial blocks,
    Reduce-Scatter -- returns this rank's shard exactly with fp32 blocks, in every policy
    (per sender / all senders) and with GPU or partial host reduction; with bf16 blocks the
    sum matches the oracle's block reduction of the same blocks;
  * the PCIe bytes each collective queues equal the volume model of Sec. 4.2.
"""
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_40093_amd as ep
from gpu_cases import TOL_MAX_ABS, TOL_MEAN_ABS, say
from paper_2609_40093_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def random_routing(rng, N, E, k):
    return np.argsort(rng.random((N, E)), axis=1)[:, :k].astype(np.int32)


def bits_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV)


@pytest.mark.parametrize("N,E,k,window", [(4096, 16, 4, (4, 8)), (3000, 64, 8, (0, 8)), (20000, 256, 8, (224, 256)),
                                          (700, 2048, 4, (1000, 1700)), (5, 8, 2, (7, 8)), (0, 8, 2, (0, 2)),
                                          (6000, 64, 8, (16, 20)), (2000, 4, 4, (2, 3))],
                         ids=["coarse_window", "first_window", "many_tiles_last_window", "wide_window",
                              "tiny", "empty", "topk_above_window_many_tiles", "one_expert_window"])
def test_window_layout_pack_partials(N, E, k, window):
    e_lo, e_hi = window
    say(f"window layout N={N} E={E} k={k} [{e_lo},{e_hi})")
    rng = np.random.default_rng(N + E)
    idx = random_routing(rng, N, E, k) if N else np.zeros((0, k), np.int32)
    want = oracle.local_layout(idx, E, e_lo, e_hi)
    lay = ep.dispatch_layout_local(torch.from_numpy(idx).to(DEV), E, e_lo, e_hi)
    torch.cuda.synchronize()
    assert np.array_equal(lay.local_counts.cpu().numpy()[:e_hi - e_lo], want.local_counts)
    assert np.array_equal(lay.local_offsets.cpu().numpy(), want.local_offsets)
    assert np.array_equal(lay.slot_pos.cpu().numpy(), want.slot_pos)
    n_local = int(want.local_offsets[-1])
    assert np.array_equal(lay.row_src.cpu().numpy()[:n_local], want.row_src)
    if N == 0:
        return
    H = 64
    x = synth.normal_bf16_rows(np.random.SeedSequence([N, 1]), N, H)
    packed = torch.zeros((max(n_local, 1), H), dtype=torch.int16, device=DEV)
    ep.pack(bits_dev(x), lay.slot_pos, packed, topk=k)
    assert np.array_equal(packed.cpu().numpy().view(np.uint16)[:n_local], x[want.row_src // k])
    # partial blocks with dyadic gates on small integers: exact
    vals = rng.integers(-40, 40, size=(max(n_local, 1), H)).astype(np.float32)
    y = (vals.view(np.uint32) >> 16).astype(np.uint16)
    w = (rng.integers(1, 8, size=(N, k)) / 8.0).astype(np.float32)
    out32 = torch.empty((N, H), dtype=torch.float32, device=DEV)
    ep.combine_rows(bits_dev(y), lay.slot_pos, torch.from_numpy(w).to(DEV), out32)
    exact, b16, _ = oracle.combine(y, want.slot_pos, w)
    assert np.array_equal(out32.cpu().numpy().astype(np.float64), exact)
    out16 = torch.empty((N, H), dtype=torch.bfloat16, device=DEV)
    ep.combine_rows(bits_dev(y), lay.slot_pos, torch.from_numpy(w).to(DEV), out16)
    assert np.array_equal(out16.view(torch.int16).cpu().numpy().view(np.uint16), b16)


@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16])
def test_combine_rows_without_rows_is_zero(out_dtype):
    """A window no token routes to: no rows, every slot -1, every sum empty."""
    say(f"combine_rows with no rows ({out_dtype})")
    N, H, k = 37, 72, 2
    slot_pos = torch.full((N * k,), -1, dtype=torch.int32, device=DEV)
    w = torch.full((N, k), 0.5, dtype=torch.float32, device=DEV)
    y = torch.empty((0, H), dtype=torch.int16, device=DEV)
    out = torch.full((N, H), 7.0, dtype=out_dtype, device=DEV)
    ep.combine_rows(y, slot_pos, w, out)
    assert torch.count_nonzero(out.float()).item() == 0


def test_window_layout_routing_errors():
    say("window layout routing errors")
    idx = np.array([[0, 1], [2, 2], [3, 0]], np.int32)       # a duplicate outside the window
    lay = ep.dispatch_layout_local(torch.from_numpy(idx).to(DEV), 4, 0, 2)
    with pytest.raises(ep.EPError, match="repeated"):
        ep.layout_validate(lay)
    idx = np.array([[0, 1], [9, 2]], np.int32)
    lay = ep.dispatch_layout_local(torch.from_numpy(idx).to(DEV), 4, 0, 2)
    with pytest.raises(ep.EPError, match="outside"):
        ep.layout_validate(lay)


def run_dense_layer(R, me, T, H, E, k, block_dtype, per_sender, on_host, rounds=2, seed=0):
    """One rank's dense layer with identity experts; returns what to check."""
    L = E // R
    rng = np.random.default_rng(seed)
    d = ep.Dense(T, H, R, self_rank=me, num_buffers=2, block_dtype=block_dtype)
    d.set_policy(per_sender=per_sender)
    peers = ep.SimPeers(d)
    peers.set_delays(inbound_us=[(r * 3001) % 2000 for r in range(R)], return_us=[(r * 7001) % 3000 for r in range(R)])
    results = []
    for rnd in range(rounds):
        buf, epoch = rnd % 2, 40 + rnd
        say(f"dense layer R={R} me={me} blocks={block_dtype} per_sender={per_sender} host={on_host} round {rnd}")
        shards = [synth.normal_bf16_rows(np.random.SeedSequence([seed, rnd, r]), T, H) for r in range(R)]
        idx_all = random_routing(rng, R * T, E, k)
        w_all = np.full((R * T, k), 1.0 / k, np.float32)
        hag = d.host_array("ag", buf)
        for r in range(R):
            if r != me:
                hag[r * T:(r + 1) * T] = shards[r]
        # peers' blocks for this rank's shard: their experts' contributions (identity experts)
        x_me = shards[me]
        idx_me = idx_all[me * T:(me + 1) * T]
        w_me = w_all[me * T:(me + 1) * T]
        blocks_in = d.host_array("rs_in", buf)
        for r in range(R):
            if r == me:
                continue
            loc = oracle.local_layout(idx_me, E, r * L, (r + 1) * L)
            y_r = x_me[loc.row_src // k] if loc.row_src.size else np.zeros((1, H), np.uint16)
            ex, b16, f32 = oracle.combine(np.ascontiguousarray(y_r), loc.slot_pos, w_me)
            blocks_in[r * T:(r + 1) * T] = f32 if block_dtype == torch.float32 else b16
        up0, down0 = d.bytes_moved()
        peers.post_dense(buf, epoch, "ag")
        ep.allgather(d, bits_dev(x_me), buf=buf, epoch=epoch)
        d.status()
        up1, down1 = d.bytes_moved()
        gathered = d.device_rows("gathered", R * T, buf).cpu().numpy().view(np.uint16)
        # grouping by this rank's experts, identity experts, partial blocks for every shard
        lay = ep.dispatch_layout_local(torch.from_numpy(idx_all).to(DEV), E, me * L, (me + 1) * L)
        n_local = int(lay.local_offsets[-1].item())
        y_local = torch.zeros((max(n_local, 1), H), dtype=torch.int16, device=DEV)
        g_dev = bits_dev(gathered)
        ep.pack(g_dev, lay.slot_pos, y_local, topk=k)
        blocks = torch.empty((R * T, H), dtype=block_dtype, device=DEV)
        ep.combine_rows(y_local, lay.slot_pos, torch.from_numpy(w_all).to(DEV), blocks)
        peers.post_dense(buf, epoch, "rs")
        out = ep.reducescatter(d, blocks, num_tokens=T, out_dtype=torch.float32, reduce_on_host=on_host, buf=buf,
                               epoch=epoch)
        d.status()
        up2, down2 = d.bytes_moved()
        hout = d.host_array("rs_out", buf)
        results.append(dict(shards=shards, gathered=gathered, out=out.cpu().numpy(), blocks=blocks.cpu(),
                            host_rs_out=np.array(hout[:R * T]), blocks_in=np.array(blocks_in[:R * T]),
                            ag_bytes=(up1 - up0, down1 - down0), rs_bytes=(up2 - up1, down2 - down1)))
    peers.drain()
    peers.close()
    d.close()
    return results


@pytest.mark.parametrize("per_sender,on_host", [(False, False), (True, False), (False, True), (True, True)],
                         ids=["all_senders_gpu_reduce", "per_sender_gpu_reduce", "all_senders_host_reduce",
                              "per_sender_host_reduce"])
def test_dense_layer_exact_f32_blocks(per_sender, on_host):
    R, me, T, H, E, k = 4, 1, 1024, 512, 16, 4
    for res in run_dense_layer(R, me, T, H, E, k, torch.float32, per_sender, on_host):
        assert np.array_equal(res["gathered"], np.concatenate(res["shards"])), "All-Gather rows differ"
        xf = (res["shards"][me].astype(np.uint32) << 16).view(np.float32)
        assert np.array_equal(res["out"], xf), "Reduce-Scatter of identity experts != own shard"
        blocks = res["blocks"].numpy()
        for r in range(R):
            if r != me:
                assert np.array_equal(res["host_rs_out"][r * T:(r + 1) * T], blocks[r * T:(r + 1) * T])
        S, Sb = T * H * 2, T * H * 4
        ag = oracle.pcie_volume("all_gather", "single_step", R, S)
        rs = oracle.pcie_volume("reduce_scatter", "cpu" if on_host else "gpu", R, Sb)
        assert res["ag_bytes"] == (ag["up"], ag["down"])
        assert res["rs_bytes"] == (rs["up"], rs["down"])


@pytest.mark.parametrize("seed", range(6))
def test_dense_layer_random_groups_exact(seed):
    """Seeded random groups (2 to 8 ranks, any self rank, either waiting policy and either
    reduction placement, token counts and row lengths): with fp32 blocks and identity
    experts the layer returns the rank's own shard exactly, the All-Gather every shard."""
    rng = np.random.default_rng(3000 + seed)
    R = int(rng.choice([2, 4, 8]))
    me = int(rng.integers(0, R))
    E = R * int(rng.choice([1, 2, 4]))
    k = int(rng.choice([kk for kk in (1, 2, 4) if kk <= E]))
    T = int(rng.integers(1, 1500))
    H = int(rng.choice([256, 512, 1024]))
    per_sender, on_host = bool(rng.integers(0, 2)), bool(rng.integers(0, 2))
    say(f"dense random group {seed}: R={R} me={me} E={E} k={k} T={T} H={H} per_sender={per_sender} host={on_host}")
    for res in run_dense_layer(R, me, T, H, E, k, torch.float32, per_sender, on_host, seed=seed):
        assert np.array_equal(res["gathered"], np.concatenate(res["shards"])), "All-Gather rows differ"
        xf = (res["shards"][me].astype(np.uint32) << 16).view(np.float32)
        assert np.array_equal(res["out"], xf), "Reduce-Scatter of identity experts != own shard"


@pytest.mark.parametrize("on_host", [False, True], ids=["gpu_reduce", "host_reduce"])
def test_dense_layer_bf16_blocks(on_host):
    """bf16 blocks: the GPU's partial blocks match the oracle's, and the Reduce-Scatter
    output matches the oracle's block reduction of the very blocks that were summed."""
    R, me, T, H, E, k = 4, 2, 512, 256, 32, 8
    res = run_dense_layer(R, me, T, H, E, k, torch.bfloat16, True, on_host, rounds=1, seed=3)[0]
    blocks = res["blocks"].view(torch.int16).numpy().view(np.uint16)
    own = oracle.bf16_to_double(blocks[me * T:(me + 1) * T])
    remote = [oracle.bf16_to_double(res["blocks_in"][r * T:(r + 1) * T]) for r in range(R) if r != me]
    if on_host:
        # the host sums the remote blocks in fp32, rank order, then rounds once to bf16
        acc = np.zeros(own.shape, np.float32)
        for blk in remote:
            acc = (acc + blk.astype(np.float32)).astype(np.float32)
        rsum = oracle.double_to_bf16(acc.astype(np.float64))
        terms = np.stack([own, oracle.bf16_to_double(rsum)])
    else:
        terms = np.stack([oracle.bf16_to_double(blocks[r * T:(r + 1) * T]) if r == me else
                          oracle.bf16_to_double(res["blocks_in"][r * T:(r + 1) * T]) for r in range(R)])
    exact, _, _ = oracle.block_reduce(terms)
    err = np.abs(res["out"].astype(np.float64) - exact)
    bound = terms.shape[0] * 2.0 ** -24 * np.abs(terms).sum(axis=0) + 1e-30
    assert np.all(err <= bound), "block reduction outside fp32 rounding of the exact sum"
    # the whole layer against the plain combine of identity experts: bf16 blocks round once more
    xf = oracle.bf16_to_double(res["shards"][me])
    d = np.abs(res["out"] - xf)
    assert d.max() <= TOL_MAX_ABS and d.mean() <= TOL_MEAN_ABS


def test_dense_per_sender_ready_ranks_land_first():
    say("dense per-sender: late rank")
    R, me, T, H = 4, 0, 2048, 1024
    d = ep.Dense(T, H, R, self_rank=me, num_buffers=1)
    d.set_policy(per_sender=True)
    peers = ep.SimPeers(d)
    peers.set_delays(inbound_us=[0, 0, 1_000_000, 0])
    x = bits_dev(synth.normal_bf16_rows(np.random.SeedSequence([9]), T, H))
    t0 = time.monotonic()
    peers.post_dense(0, 5, "ag")
    ep.allgather(d, x, epoch=5)
    landed = d.host_array("ag_landed")
    t_end = t0 + 5.0
    while not (landed[1] == 5 and landed[3] == 5) and time.monotonic() < t_end:
        time.sleep(0.0005)
    assert landed[1] == 5 and landed[3] == 5 and landed[2] != 5 and time.monotonic() - t0 < 1.0
    d.status()
    peers.drain()
    peers.close()
    d.close()


def test_set_policy_while_a_host_reduction_is_pending():
    """ep_dense_set_policy called over and over while a Reduce-Scatter with partial host
    reduction is pending (its ranks' blocks arrive 0.2 s late, then the host sums them):
    each call waits for a reduction in progress instead of stopping its threads, and the
    round's result is exact (dyadic blocks, fp32)."""
    R, me, T, H = 4, 1, 1024, 512
    say("dense set_policy during a pending host reduction")
    d = ep.Dense(T, H, R, self_rank=me, num_buffers=1, block_dtype=torch.float32)
    d.set_policy(per_sender=False, host_threads=4)
    peers = ep.SimPeers(d)
    peers.set_delays(inbound_us=[0] * R, return_us=[200_000] * R)
    rng = np.random.default_rng(12)
    blocks_h = (rng.integers(-64, 64, size=(R * T, H)) / 8).astype(np.float32)
    rs_in = d.host_array("rs_in")
    want = blocks_h[me * T:(me + 1) * T].copy()
    for r in range(R):
        if r != me:
            blk = (rng.integers(-64, 64, size=(T, H)) / 8).astype(np.float32)
            rs_in[r * T:(r + 1) * T] = blk
            want += blk                                  # multiples of 1/8 below 64: exact
    blocks = torch.from_numpy(blocks_h).to(DEV)
    peers.post_dense(0, 7, "rs")
    out = ep.reducescatter(d, blocks, num_tokens=T, out_dtype=torch.float32, reduce_on_host=True, epoch=7)
    t_end = time.monotonic() + 0.5
    n = 0
    while time.monotonic() < t_end:
        d.set_policy(per_sender=False, host_threads=2 + n % 4)
        n += 1
        time.sleep(0.001)
    d.status()
    assert np.array_equal(out.cpu().numpy(), want)
    peers.drain()
    peers.close()
    d.close()
