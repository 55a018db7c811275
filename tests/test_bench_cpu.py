"""bench.py's host logic on the CPU: the algorithmic bytes behind every roofline figure,
the pair roofline, the committed counter figures' freshness check, and the one-GPU rule."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2609_40093_amd import synth  # noqa: E402

# Bytes each kernel must move per layer, in MB (1e6), for the five workloads: the figures
# of the hot-path scope table, worked out from the definitions (pack reads each token row
# once and writes its k copies plus the slot positions; combine reads the k rows, gates
# and slot positions and writes one row per token).
EXPECTED_MB = {
    "tiny": (0.787, 0.788),
    "coarse": (100.7, 100.7),
    "fine": (302.3, 302.5),
    "decode": (33.0, 33.0),
    "prefill": (4229.0, 4230.0),
}


@pytest.mark.parametrize("name", sorted(EXPECTED_MB))
def test_algorithmic_bytes_match_the_scope_table(name):
    cfg = synth.config(name)
    b = bench.algorithmic_bytes(cfg)
    pack_mb, combine_mb = EXPECTED_MB[name]
    digits = 3 if pack_mb < 1 else (1 if pack_mb < 1000 else 0)
    assert round(b["pack"] / 1e6, digits) == pack_mb
    assert round(b["combine"] / 1e6, digits) == combine_mb
    n = cfg.T * cfg.k
    assert b["layout_pack"] == b["pack"] + 8 * n        # plus reading the ids and writing row_src
    assert b["layout"] == 12 * n


def test_pair_roofline_sums_bytes_and_time():
    kernels = {"layout_pack": {"algorithmic_bytes": 100, "avg_us": 1e-3},
               "combine": {"algorithmic_bytes": 300, "avg_us": 3e-3}}
    r = bench.pair_roofline(kernels)
    assert r["kernels"] == ["layout_pack", "combine"]
    assert r["algorithmic_bytes"] == 400 and r["avg_us"] == pytest.approx(4e-3)
    assert r["achieved"] == pytest.approx(100.0) and r["frac"] == pytest.approx(100.0 / bench.HBM_PEAK_GBPS)
    two = {"pack": kernels["layout_pack"], "combine": kernels["combine"]}
    assert bench.pair_roofline(two)["kernels"] == ["pack", "combine"]


TRAFFIC_FILES = sorted(f for f in os.listdir(os.path.join(ROOT, "profiles"))
                       if f.startswith("traffic_") and f.endswith(".json"))


@pytest.mark.parametrize("fname", TRAFFIC_FILES)
def test_committed_traffic_is_fresh_and_close_to_the_definition(fname, monkeypatch):
    """A committed counter figure is used only while the kernel's sources hash as when it
    was taken; when used, it is within 2% of the algorithmic bytes (no wasted re-reads), or,
    for the layout, within twice its bytes plus a fixed 256 KiB per launch."""
    rec = json.load(open(os.path.join(ROOT, "profiles", fname)))
    kernel, workload = rec["kernel"], rec["workload"]
    assert fname == f"traffic_{kernel}_{workload}.json"
    traffic = bench.committed_traffic(workload, kernel)
    if traffic is None:
        pytest.skip("the kernel changed since its counters were taken (the bench reports null)")
    want = bench.algorithmic_bytes(synth.config(workload))[kernel]
    if kernel == "layout":
        # latency-bound, two kernels that each read the routing ids, plus a fixed cost per
        # launch (code and arguments fetched into each XCD's L2) that shows on small layouts
        assert traffic <= 2 * want + (256 << 10)
    else:
        assert abs(traffic - want) <= 0.02 * want
    assert rec["source_sha256"] == bench.source_hash(kernel)
    monkeypatch.setattr(bench, "source_hash", lambda k: "0" * 16)
    assert bench.committed_traffic(workload, kernel) is None


def test_kernel_hash_covers_its_headers(tmp_path, monkeypatch):
    """The hash changes with any file the kernel is compiled from, headers included."""
    csrc = tmp_path / "paper_2609_40093_amd" / "csrc"
    csrc.mkdir(parents=True)
    for name in bench.KERNEL_SOURCES["layout_pack"]:
        (csrc / name).write_text(name)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.source_hash("layout_pack")
    (csrc / "wave.h").write_text("changed")
    assert bench.source_hash("layout_pack") != h0


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_a_failed_pinned_mode_reports_its_flag_words():
    """bench.staging_flags reads every host flag word of each buffer set (absent kinds: None)."""
    import ctypes
    import types
    send, recv = (ctypes.c_uint32 * 2)(5, 6), (ctypes.c_uint32 * 3)(1, 2, 3)
    landed = (ctypes.c_uint32 * 3)(7, 0, 7)
    v = types.SimpleNamespace(num_ranks=3, max_chunks=2, mode=9, send_flags=ctypes.addressof(send),
                              recv_flags=ctypes.addressof(recv), in_flags=None, ret_flags=None, in_landed=None,
                              recv_landed=ctypes.addressof(landed))
    got = bench.staging_flags(types.SimpleNamespace(views=[v]))
    assert got == {"0": {"mode": 9, "send": [5, 6], "recv": [1, 2, 3], "in": None, "ret": None, "in_landed": None,
                         "recv_landed": [7, 0, 7]}}


def test_cpu_baseline_reports_all_cores_and_one():
    """The CPU baseline times the oracle on whole layers on every core this process may use
    and on one thread, and names the host's CPU model."""
    cfg = synth.config("tiny")
    inp = synth.make_inputs(cfg)
    r = bench.cpu_baseline(cfg, inp, inp.expert_outputs(), 0.2)
    assert r["kind"] == "oracle" and r["unit"] == "GB/s" and r["value"] > 0
    assert r["cores"] == len(os.sched_getaffinity(0)) == r["cores_available"]
    assert r["single_thread"]["cores"] == 1 and r["single_thread"]["value"] > 0
    assert r["cpu_model"] and "whole tiny layer" in r["sample"]


def test_default_workload_is_the_prefill_layer():
    assert bench.parse.__defaults__ is None
    old = sys.argv
    try:
        sys.argv = ["bench.py"]
        assert bench.parse().workload == "prefill"
    finally:
        sys.argv = old


def test_pattern_bound_takes_the_slowest_direction_of_each_phase():
    peaks = {"d2h_alone": 50.0, "h2d_alone": 40.0, "both": 80.0}   # GB/s
    # one phase up only: 1 GB at 50 GB/s = 20 ms
    assert bench.pattern_bound_us([(1e9, 0)], peaks) == pytest.approx(20000.0)
    # both ways at once: 1 GB up, 3 GB down -> the download (75 ms) bounds it, not 4 GB / 80
    assert bench.pattern_bound_us([(1e9, 3e9)], peaks) == pytest.approx(75000.0)
    # equal both ways: the two-way peak bounds it (2 GB / 80 = 25 ms > 1 GB / 40 = 25 ms)
    assert bench.pattern_bound_us([(1e9, 1e9)], peaks) == pytest.approx(25000.0)
    # phases add up
    assert bench.pattern_bound_us([(1e9, 0), (0, 1e9)], peaks) == pytest.approx(20000.0 + 25000.0)


def test_streaming_ceiling_takes_the_faster_store_policy_of_the_kernels_mix():
    ceil = {"write_only": {"frac": 0.68}, "write_only_write_through": {"frac": 0.69},
            "write_only_write_through_nt": {"frac": 0.685},
            "combine_like_8_to_1": {"frac": 0.73}, "combine_like_8_to_1_write_through": {"frac": 0.70},
            "combine_like_8_to_1_write_through_nt": {"frac": 0.69}, "note": "probe"}
    got = bench.ceiling_of("pack", 0.69, ceil, 8)
    assert got["mix"] == "write_only_write_through" and got["frac"] == 0.69 and got["kernel_frac_of_ceiling"] == 1.0
    ceil["write_only_write_through_nt"] = {"frac": 0.70}
    got = bench.ceiling_of("pack", 0.69, ceil, 8)
    assert got["mix"] == "write_only_write_through_nt" and got["kernel_frac_of_ceiling"] == round(0.69 / 0.70, 3)
    got = bench.ceiling_of("combine", 0.711, ceil, 8)
    assert got["mix"] == "combine_like_8_to_1" and got["kernel_frac_of_ceiling"] == round(0.711 / 0.73, 3)
    assert "note" in bench.ceiling_of("layout_pack", 0.69, {"note": "no instance"}, 2)
