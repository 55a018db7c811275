"""bench.py's pinned section on the GPU: a mode whose flag waits expire is recorded with its
error and its flag words, and the other modes still run.  The expiry is forced from the host:
the simulated peers of that mode never answer, and its waits are bounded at 20 ms."""
import os
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

torch = pytest.importorskip("torch")

import bench  # noqa: E402
import paper_2609_40093_amd as ep  # noqa: E402
from paper_2609_40093_amd import synth  # noqa: E402


@pytest.mark.gpu
def test_a_failed_pinned_mode_is_recorded_and_the_others_run(monkeypatch):
    print("[gpu] bench pinned section with one mode's peers withheld (tiny layer)", flush=True)
    cfg = synth.config("tiny")
    inp = synth.make_inputs(cfg)
    args = types.SimpleNamespace(steps=10, warmup=2, chunk_mib=16, workload="tiny")
    monkeypatch.setattr(bench, "PINNED_MODES", (("per_sender", 1), ("default", 0)))
    set_mode, post = ep.Staging.set_mode, ep.SimPeers.post

    def set_mode_bounded(self, mode, self_rank=0):
        set_mode(self, mode, self_rank)
        self.set_wait(timeout_us=20_000, sleep_units=1)
        self.withheld = True

    def post_unless_withheld(self, buf, epoch, rows, delay_us=0):
        if not getattr(self.staging, "withheld", False):
            post(self, buf, epoch, rows, delay_us)

    monkeypatch.setattr(ep.Staging, "set_mode", set_mode_bounded)
    monkeypatch.setattr(ep.SimPeers, "post", post_unless_withheld)
    r = bench.bench_pinned(cfg, inp, inp.expert_outputs(), args, torch.device("cuda", 0))
    failed = r["modes"]["per_sender"]
    assert "EP_ERR_TIMEOUT" in failed["error"], failed["error"]
    assert set(failed["flags"]) == {"0", "1"} and failed["flags"]["0"]["mode"] == 1
    assert len(failed["flags"]["0"]["recv"]) == cfg.R
    ok = r["modes"]["default"]
    assert "error" not in ok and ok["us_per_layer"] > 0
    assert "error" not in r["dense_allgather_reducescatter"]


@pytest.mark.gpu
def test_bench_runs_end_to_end_on_the_tiny_layer():
    """The HBM-staged part of bench.py on the tiny layer in a process of its own: one JSON
    line with the value, the roofline of the dispatch and combine kernels, and the same
    steps replayed from a HIP graph."""
    import json
    import subprocess
    print("[gpu] bench.py --workload tiny --no-pinned --no-cpu-baseline", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--no-pinned",
                        "--no-cpu-baseline", "--steps", "20", "--warmup", "3"], capture_output=True, text=True,
                       timeout=240)
    assert r.returncode == 0, r.stderr[-3000:]
    d = json.loads(r.stdout.strip().splitlines()[-1])
    assert d["value"] > 0 and d["n_gpus"] == 1 and d["config"]["T"] == 128
    assert d["roofline"]["bound"] == "hbm" and d["roofline"]["frac"] > 0
    g = d["graph_replayed_steps"]
    assert "error" not in g, g
    assert g["us_per_layer"] > 0 and g["steps"] >= 20
