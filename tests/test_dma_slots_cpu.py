"""The SDMA legs' signal handling on the host, against a stand-in ROCr runtime
(tests/host/dma_slots_test.cpp): no GPU, no HIP.

The stand-in keeps the documented contract of an async copy (it starts once every
dependency signal reads 0, and decrements its completion signal after its bytes are
visible) and applies decrements late, after the flag the copy wrote can already be seen.
It records a violation when a decrement lands on a signal that was reset or destroyed
since, or when a dependency drops below 0 (an engine would then never start the copy).

Cases:
- lane: rounds of the default device->host leg with the chunk count changing between
  rounds (signal roles shift), lanes created and released between batches, the chunk
  flags on the data engine or on an engine of their own;
- exchange: calls with outbound and inbound copies (courier, per-sender and all-senders
  jobs), senders answering in random order, exchanges recreated between batches, the
  flags on the data engines or on two flag engines, the landed flags of merged inbound
  copies as one flag copy from an epoch row;
- order: a later call's sender answers before an earlier call's; both calls finish
  without waiting for the bound (the courier serves jobs in call order);
- merge: inbound copies contiguous in memory whose senders have answered go down as one
  data copy with each sender's flag after it (one flag copy for flags in neighbouring
  words when the job has an epoch row); a rank's own rows (an eager copy) go down
  before the other senders of an all-senders job answer; the pieces of a host-side result
  (eager copies whose flags the job's host work raises) go down as each is ready, without
  their flags holding back that host work;
- graph: 200 graph-replayed rounds with SDMA legs (graph_legs.h) between a device
  stand-in and simulated peers, with the row count changing from round to round: every
  send flag comes after its rows, every landed word after the returned rows;
- graph_timeout: the same thread with peers that never answer records the expired wait
  (site, flag, round) in the status block and still lands the round; a stop ends its wait
  for a round the device never reaches;
- bounded: a slot with a signal that never retires is refused after its bound, with a
  message; a failed copy (negative value) is reported once; nothing is destroyed while a
  decrement may still come;
- the lane, exchange, order, merge and graph scenarios again, built with ThreadSanitizer: no
  data race between the courier thread, the graph legs' thread, the stand-in engines and
  the callers' threads;
- old_rule: the reuse rule of the earlier revision (a completion signal shared by two
  copies, reset as soon as the flags are seen) replayed against the stand-in, which must
  report the late decrement: the harness does catch the failure mode.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_40093_amd", "csrc")
ROCM_INCLUDE = "/opt/rocm/include"


@pytest.fixture(scope="module")
def binary(tmp_path_factory):
    gxx = shutil.which("g++")
    if not gxx or not os.path.exists(os.path.join(ROCM_INCLUDE, "hsa", "hsa.h")):
        pytest.skip("needs g++ and the ROCr headers")
    out = str(tmp_path_factory.mktemp("dma") / "dma_slots_test")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE,
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host", "dma_slots_test.cpp"), os.path.join(CSRC, "sdma_lane.cpp"),
           os.path.join(CSRC, "graph_legs.cpp"),
           "-o", out, "-lpthread"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-4000:]
    return out


def run(binary, *args, timeout=120):
    res = subprocess.run([binary, *map(str, args)], capture_output=True, text=True, timeout=timeout)
    return res.returncode, res.stdout + res.stderr


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_lane_rounds_never_reset_a_pending_signal(binary, seed):
    rc, out = run(binary, "lane", seed)
    assert rc == 0, out
    assert "violations 0 checks_failed 0" in out


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_exchange_calls_never_reset_a_pending_signal(binary, seed):
    rc, out = run(binary, "exchange", seed)
    assert rc == 0, out
    assert "violations 0 checks_failed 0" in out


def test_senders_out_of_call_order_do_not_stall_the_inbound_engine(binary):
    rc, out = run(binary, "order", timeout=60)
    assert rc == 0, out


def test_contiguous_ready_copies_go_as_one_and_own_rows_go_first(binary):
    rc, out = run(binary, "merge", timeout=60)
    assert rc == 0, out


@pytest.mark.parametrize("seed", [1, 2])
def test_graph_legs_raise_flags_only_after_their_rows(binary, seed):
    rc, out = run(binary, "graph", seed)
    assert rc == 0, out
    assert "violations 0 checks_failed 0" in out


def test_graph_legs_report_an_expired_wait_and_stop(binary):
    rc, out = run(binary, "graph_timeout", timeout=60)
    assert rc == 0, out


def test_slot_reuse_is_bounded_and_reported(binary):
    rc, out = run(binary, "bounded", timeout=60)
    assert rc == 0, out


def test_harness_catches_the_shared_signal_rule(binary):
    rc, out = run(binary, "old_rule", 1, timeout=60)
    assert rc == 1, out
    assert "decrement landed after the signal was reset" in out


@pytest.fixture(scope="module")
def tsan_binary(tmp_path_factory):
    """The same harness built with ThreadSanitizer (host code only: g++, no GPU code)."""
    gxx = shutil.which("g++")
    if not gxx or not os.path.exists(os.path.join(ROCM_INCLUDE, "hsa", "hsa.h")):
        pytest.skip("needs g++ and the ROCr headers")
    out = str(tmp_path_factory.mktemp("dma_tsan") / "dma_slots_test_tsan")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=thread", "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE,
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host", "dma_slots_test.cpp"), os.path.join(CSRC, "sdma_lane.cpp"),
           os.path.join(CSRC, "graph_legs.cpp"),
           "-o", out, "-lpthread"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0 and "tsan" in (res.stderr + res.stdout).lower():
        pytest.skip("ThreadSanitizer runtime not available: " + res.stderr[-300:])
    assert res.returncode == 0, res.stderr[-4000:]
    return out


@pytest.mark.parametrize("scenario", ["lane", "exchange", "order", "merge", "graph"])
def test_lane_courier_and_slots_have_no_data_race(tsan_binary, scenario):
    """The lane, the courier thread, the signal slots and the callers' threads share flags,
    signals and job queues: ThreadSanitizer reports no data race in any scenario."""
    rc, out = run(tsan_binary, scenario, 2, timeout=300)
    assert "ThreadSanitizer" not in out, out[-4000:]
    assert rc == 0 and "violations 0 checks_failed 0" in out, out[-2000:]
