"""Host-staged dispatch/combine on the GPU: SDMA legs, completion flags in pinned host
memory, the bounded flag wait, and the simulated peers.

Every wait here is bounded: flags that are withheld are withheld with a short
timeout, so the wait kernel records a timeout and exits normally."""
import threading
import time

import numpy as np
import pytest
import torch

import paper_2609_40093_amd as ep
from gpu_cases import (TOL_MAX_ABS, TOL_MEAN_ABS, combine_errors, from_config, make_case,
                       oracle_reference, say)

pytestmark = pytest.mark.gpu

DEV = "cuda"


def dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV)


def layout_of(case):
    lay = ep.dispatch_layout(torch.from_numpy(case.topk_idx).to(DEV), case.E, case.R)
    ep.layout_validate(lay)
    return lay


@pytest.mark.parametrize("chunk", [4096, 1 << 20, 0])
def test_dispatch_host_bytes_and_flags(chunk):
    case = make_case("pinned_dispatch", 1000, 1032, 32, 4, 4, "random", seed=1)
    say(f"pinned dispatch chunk={chunk}")
    ref_lay, packed, _, _, _ = oracle_reference(case)
    st = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=2, chunk_bytes=chunk)
    lay = layout_of(case)
    ep.dispatch(dev_bits(case.x), lay.slot_pos, st, topk=case.k, buf=1, epoch=7)
    st.status()
    host = st.host_array("send", 1)[:case.slots]
    assert host.tobytes() == packed.tobytes(), "host bounce buffer differs from the oracle's packed rows"
    nbytes = case.slots * st.row_bytes
    used = -(-nbytes // st.chunk_bytes)
    flags = st.host_array("send_flags", 1)
    assert (flags[:used] == 7).all() and (flags[used:] == 0).all()
    assert (st.host_array("send_flags", 0) == 0).all()       # the other buffer set is untouched
    st.close()


def test_combine_from_host_matches_hbm_and_oracle():
    case = from_config("decode")     # 256 tokens x 7168, 256 experts top-8, 8 ranks
    say("pinned combine, decode-shaped layer")
    ref_lay, _, exact, _, _ = oracle_reference(case)
    lay = layout_of(case)
    w = torch.from_numpy(case.topk_w).to(DEV)
    pin = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=1)
    pin.host_array("recv", 0)[:case.slots] = case.y
    pin.host_array("recv_flags", 0)[:] = 3
    out_pin = ep.combine(pin, lay.slot_pos, w, epoch=3)
    pin.status()
    hbm = ep.Staging("hbm", case.slots, case.H, case.R, num_buffers=1)
    hbm.write_device("recv", dev_bits(case.y))
    out_hbm = ep.combine(hbm, lay.slot_pos, w)
    torch.cuda.synchronize()
    assert torch.equal(out_pin.view(torch.int16), out_hbm.view(torch.int16))
    mx, mean = combine_errors(out_pin.view(torch.int16).cpu().numpy().view(np.uint16), exact)
    assert mx <= TOL_MAX_ABS and mean <= TOL_MEAN_ABS
    pin.close()
    hbm.close()


def test_stale_epoch_is_not_consumed():
    case = make_case("stale", 64, 256, 16, 2, 4, "random", seed=2)
    say("stale epoch -> bounded wait times out")
    lay = layout_of(case)
    w = torch.from_numpy(case.topk_w).to(DEV)
    st = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=1)
    st.set_wait(timeout_us=2000, sleep_units=1)
    st.host_array("recv", 0)[:case.slots] = case.y
    st.host_array("recv_flags", 0)[:] = 4           # last round's epoch
    ep.combine(st, lay.slot_pos, w, epoch=5)
    with pytest.raises(ep.EPError) as ei:
        st.status()
    assert ei.value.status == 5                      # EP_ERR_TIMEOUT
    # the message names the wait, the flag it gave up on, what it read and what it wanted
    msg = str(ei.value)
    assert "wait_recv gave up on recv_flags[buf 0][rank " in msg, msg
    assert "last read 4 (waited for 5)" in msg, msg
    st.status()                                      # the status block was cleared
    st.host_array("recv_flags", 0)[:] = 5
    st.set_wait(timeout_us=5_000_000)
    out = ep.combine(st, lay.slot_pos, w, epoch=5)
    st.status()
    _, _, exact, _, _ = oracle_reference(case)
    mx, mean = combine_errors(out.view(torch.int16).cpu().numpy().view(np.uint16), exact)
    assert mx <= TOL_MAX_ABS and mean <= TOL_MEAN_ABS
    st.close()


def test_wait_sees_flags_raised_later():
    """The polling lanes pick up host writes made after the combine was enqueued."""
    case = make_case("late_flags", 200, 512, 16, 2, 4, "random", seed=4)
    say("late flags from a host thread")
    lay = layout_of(case)
    w = torch.from_numpy(case.topk_w).to(DEV)
    st = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=1)
    st.set_wait(timeout_us=20_000_000)
    st.host_array("recv", 0)[:case.slots] = case.y
    flags = st.host_array("recv_flags", 0)

    def raise_flags():
        for r in range(case.R):
            time.sleep(0.01)
            flags[r] = 9

    th = threading.Thread(target=raise_flags)
    t0 = time.time()
    out = ep.combine(st, lay.slot_pos, w, epoch=9)
    th.start()
    st.status()
    th.join()
    assert time.time() - t0 >= 0.03
    _, _, exact, _, _ = oracle_reference(case)
    mx, mean = combine_errors(out.view(torch.int16).cpu().numpy().view(np.uint16), exact)
    assert mx <= TOL_MAX_ABS and mean <= TOL_MEAN_ABS
    st.close()


def test_echo_rounds_alternating_buffers():
    """Dispatch -> simulated peers echo the rows through host memory -> combine, for
    several rounds over two buffer sets: with identity experts and dyadic gates every
    round returns x exactly."""
    case = make_case("echo", 3000, 2048, 128, 8, 8, "skewed", seed=6, gates="uniform")
    say("echo rounds through host memory")
    lay = layout_of(case)
    w = torch.from_numpy(case.topk_w).to(DEV)
    x = dev_bits(case.x)
    st = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=2, chunk_bytes=4 << 20)
    peers = ep.SimPeers(st, echo=True)
    outs = []
    for rnd in range(4):
        buf, epoch = rnd % 2, rnd + 1
        ep.dispatch(x, lay.slot_pos, st, topk=case.k, buf=buf, epoch=epoch)
        peers.post(buf, epoch, case.slots)
        outs.append(ep.combine(st, lay.slot_pos, w, out_dtype=torch.float32, buf=buf, epoch=epoch))
    st.status()
    peers.drain()
    xf = torch.from_numpy(case.x.view(np.int16)).view(torch.bfloat16).float()
    for o in outs:
        assert torch.equal(o.cpu(), xf)
    peers.close()
    st.close()


def test_coarse_layer_pinned_with_peers():
    """The 4096-token coarse-expert layer, host-staged end to end with flag-only peers."""
    case = from_config("coarse")
    say("coarse layer, pinned, sim peers")
    ref_lay, packed, exact, _, _ = oracle_reference(case)
    lay = layout_of(case)
    w = torch.from_numpy(case.topk_w).to(DEV)
    st = ep.Staging("pinned", case.slots, case.H, case.R, num_buffers=1)
    st.host_array("recv", 0)[:case.slots] = case.y
    peers = ep.SimPeers(st, echo=False)
    ep.dispatch(dev_bits(case.x), lay.slot_pos, st, topk=case.k, epoch=11)
    peers.post(0, 11, case.slots)
    out = ep.combine(st, lay.slot_pos, w, epoch=11)
    st.status()
    peers.drain()
    assert st.host_array("send", 0)[:case.slots].tobytes() == packed.tobytes()
    mx, mean = combine_errors(out.view(torch.int16).cpu().numpy().view(np.uint16), exact)
    assert mx <= TOL_MAX_ABS and mean <= TOL_MEAN_ABS
    peers.close()
    st.close()


def test_free_waits_for_the_host_leg_in_flight():
    """ep_staging_free right after a dispatch whose SDMA upload (128 MiB, several ms over
    PCIe) is still running: the free waits for the copies to land before it frees their
    buffers, so pinned memory allocated right after keeps what is written into it, and a
    new staging runs a correct round."""
    T, H, E, k, R = 8192, 4096, 8, 2, 4
    case = make_case("free_in_flight", T, H, E, k, R, "random", seed=6)
    say("free a pinned staging while its host leg is in flight")
    _, packed, _, _, _ = oracle_reference(case)
    lay = layout_of(case)
    x = dev_bits(case.x)
    st = ep.Staging("pinned", case.slots, H, R, num_buffers=1, chunk_bytes=1 << 20)
    ep.dispatch(x, lay.slot_pos, st, topk=k, buf=0, epoch=9)
    t0 = time.monotonic()
    st.close()
    assert time.monotonic() - t0 < 6.0
    fresh = torch.full((case.slots * H,), 0x5A5A, dtype=torch.int16, pin_memory=True)
    time.sleep(0.02)
    assert bool((fresh == 0x5A5A).all()), "pinned memory changed after the staging was freed"
    del fresh
    st2 = ep.Staging("pinned", case.slots, H, R, num_buffers=1, chunk_bytes=1 << 20)
    ep.dispatch(x, lay.slot_pos, st2, topk=k, buf=0, epoch=1)
    st2.status()
    assert st2.host_array("send", 0)[:case.slots].tobytes() == packed.tobytes()
    st2.close()


def test_free_after_an_unanswered_exchange_round():
    """A duplex dispatch whose senders never raise their flags (no peers, a 0.3 s wait):
    the wait expires normally, and freeing the staging then queues the inbound copies the
    library still holds and waits for them to land; a new staging runs a correct round."""
    T, H, E, k, R, me = 512, 1024, 16, 2, 4, 1
    case = make_case("unanswered", T, H, E, k, R, "random", seed=8)
    say("free after an exchange round nobody answered")
    _, packed, _, _, _ = oracle_reference(case)
    lay = layout_of(case)
    x = dev_bits(case.x)
    st = ep.Staging("pinned", case.slots, H, R, num_buffers=1, chunk_bytes=1 << 20)
    st.set_mode(ep.MODE_DUPLEX | ep.MODE_PER_SENDER, self_rank=me)
    st.set_wait(timeout_us=300_000, sleep_units=1)
    st.set_inbound(0, [0 if r == me else 64 for r in range(R)])
    ep.dispatch(x, lay.slot_pos, st, topk=k, buf=0, epoch=3, rank_offsets=lay.rank_offsets)
    t0 = time.monotonic()
    st.close()
    assert time.monotonic() - t0 < 8.0
    st2 = ep.Staging("pinned", case.slots, H, R, num_buffers=1, chunk_bytes=1 << 20)
    ep.dispatch(x, lay.slot_pos, st2, topk=k, buf=0, epoch=1)
    st2.status()
    assert st2.host_array("send", 0)[:case.slots].tobytes() == packed.tobytes()
    st2.close()
