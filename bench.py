"""Benchmark of one rank's MoE dispatch + combine on one MI355X.

A step is one MoE layer's communication share: dispatch layout, pack, and the
gate-weighted combine of the returned rows (the peers' expert outputs are seeded data
already in the receive buffer).  Layout and pack are one call (ep_dispatch_fused), which
runs them as one kernel when the layer has few experts (as the headline layer does) and
as two kernels otherwise; the two-kernel path is also timed, for comparison.  `value` is token payload throughput with HBM staging:
(dispatch payload + combine payload) / layer time, each payload T*k*2H bytes.  The same
layer with pinned host staging (SDMA legs, host flags, simulated peers) is timed after
it and reported under "pinned_staging"; that rate includes PCIe and is never `value`.

Inputs and staging are rotated over enough buffer sets that each step's working set
has left the 256 MB Infinity Cache before it is used again.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "dispatch & combine GB/s token payload (μs/MoE layer) + % HBM/PCIe roofline, 1 GPU"
HBM_PEAK_GBPS = 8000.0      # MI355X HBM3E
PCIE_PEAK_GBPS = 64.0       # PCIe Gen5 x16, per direction
MALL_BYTES = 256 << 20
SPIN_CYCLES = 240_000       # a device spin of about 100 us at 2.4 GHz (torch.cuda._sleep)
_T0 = time.perf_counter()


def progress(msg: str) -> None:
    """One line on stderr as each part of the run ends (the JSON line alone goes to stdout)."""
    print(f"[bench +{time.perf_counter() - _T0:6.1f}s] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="prefill",
                   help="synth config name (default: the large prefill layer, T=32768, H=7168, top-8 of 256)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-pinned", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="least host time spent on each CPU-baseline figure (whole layers only)")
    p.add_argument("--chunk-mib", type=int, default=16, help="device->host DMA chunk of the pinned legs")
    return p.parse_args()


def algorithmic_bytes(cfg) -> dict:
    """Bytes each kernel must move per launch (reads + writes), per the path's definition."""
    T, H, k = cfg.T, cfg.H, cfg.k
    n = T * k
    row = 2 * H
    out = {
        "pack": T * row + n * row + 4 * n,                  # read x once, write k copies, read slot_pos
        "combine": n * row + 8 * n + T * row,               # read k rows, gates and slot_pos, write out
        "layout": 4 * n + 4 * n + 4 * n,                    # read ids, write slot_pos and row_src
    }
    # one kernel: read ids and x once, write k copies, slot_pos and row_src
    out["layout_pack"] = T * row + n * row + 4 * n + 4 * n + 4 * n
    return out


# the files each kernel is compiled from: its source and the package headers it includes
KERNEL_SOURCES = {"pack": ("pack.hip", "ep_internal.h"), "combine": ("combine.hip", "ep_internal.h"),
                  "layout": ("layout.hip", "wave.h", "ep_internal.h"),
                  "layout_pack": ("fused.hip", "wave.h", "ep_internal.h")}
TIMED_KERNELS = ("layout_pack", "pack", "combine")


def source_hash(kernel: str) -> str:
    """Hash of the files the kernel is compiled from (a change to any of them makes the
    committed counter figures stale)."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, "paper_2609_40093_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def committed_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken
    on the kernel source as it is now (else None)."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    d = json.load(open(path))
    if kernel not in KERNEL_SOURCES or d.get("source_sha256") != source_hash(kernel):
        return None
    return d.get("traffic_bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU: the path is one rank's share "
                                   "of an expert-parallel group, simulated on a single MI355X; "
                                   f"--gpus {args.gpus} is not supported"}))
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2609_40093_amd as ep
    from paper_2609_40093_amd import _lib, synth

    _lib.load()                                        # fails loudly if libep.so is missing
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    cfg = synth.config(args.workload)
    inp = synth.make_inputs(cfg)
    y = inp.expert_outputs()
    progress(f"{cfg.name} layer inputs generated")
    T, H, E, k, R = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R
    n = cfg.slots
    payload = cfg.payload_bytes
    step_bytes = 2 * payload + T * 2 * H * 2   # x, packed, recv, out per set (for rotation sizing)
    nsets = max(2, min(8, -(-3 * MALL_BYTES // step_bytes) + 1))
    stream = torch.cuda.current_stream()

    x_d = torch.from_numpy(inp.x.view(np.int16)).to(dev)
    idx_d = torch.from_numpy(inp.topk_idx).to(dev)
    w_d = torch.from_numpy(inp.topk_w).to(dev)
    y_d = torch.from_numpy(y.view(np.int16)).to(dev)
    sets = []
    for s in range(nsets):
        sets.append(dict(x=x_d.clone(), idx=idx_d.clone(), w=w_d.clone(),
                         out=torch.empty((T, H), dtype=torch.bfloat16, device=dev), lay=None))
    staging = ep.Staging("hbm", n, H, R, num_buffers=nsets)
    for s in range(nsets):
        staging.write_device("recv", y_d, buf=s)
    torch.cuda.synchronize()

    def step(i, trace=None, fused=True):
        """One layer; `trace` names the call ("dispatch", "combine" or "both") whose kernels
        are bracketed by timing events.  fused=False: layout and dispatch as two calls."""
        st = sets[i % nsets]
        if trace in ("dispatch", "both"):
            ep.trace_enable(True)
        if fused:
            st["lay"] = ep.dispatch_fused(st["x"], st["idx"], E, R, staging, buf=i % nsets, epoch=i + 1,
                                          out=st["lay"])
        else:
            st["lay"] = ep.dispatch_layout(st["idx"], E, R, out=st["lay"])
            ep.dispatch(st["x"], st["lay"].slot_pos, staging, topk=k, buf=i % nsets, epoch=i + 1)
        if trace == "dispatch":
            ep.trace_enable(False)
        elif trace == "combine":
            ep.trace_enable(True)
        ep.combine(staging, st["lay"].slot_pos, st["w"], out=st["out"], buf=i % nsets, epoch=i + 1)
        if trace in ("combine", "both"):
            ep.trace_enable(False)

    # ---- HBM staging: warmup, then exactly K timed steps; the dispatch and combine
    #      kernels are timed live with HIP events on the stream they run on
    for i in range(args.warmup):
        step(i)
    ep.layout_validate(sets[0]["lay"])
    torch.cuda.synchronize()
    probe0 = time.perf_counter()
    step(args.warmup)
    torch.cuda.synchronize()
    probe_us = (time.perf_counter() - probe0) * 1e6
    # A launch bracketed by timing events costs the stream about 4 us and the host 10-25 us
    # (binding the start event to the kernel).  On layers of a few hundred us or more the
    # timed steps carry them, the dispatch's kernels on one step and the combine's on the
    # next (about 0.4% of the step; the host stays far ahead of the device); shorter layers
    # would become bound by that host time, so their timed steps run without events and the
    # kernel averages come from the breakdown pass.
    every = probe_us > 300.0
    ep.trace_reset()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(args.warmup + i, trace=("dispatch", "combine")[i % 2] if every else None)
    t_issue = time.perf_counter()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    timed_stats = ep.trace_read()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    progress(f"{args.steps} timed steps: {ms_per_step * 1e3:.1f} us per layer")
    value = 2 * payload / (ms_per_step * 1e-3) / 1e9
    issue_us = (t_issue - t0) * 1e6 / args.steps
    # warm cache, beside the headline: every step on buffer set 0 (inputs and staging
    # stay in the 256 MB memory-side cache between steps); meaningless when one set is
    # larger than that cache
    warm = None
    if step_bytes < MALL_BYTES:
        for i in range(args.warmup):
            step(i * nsets)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for i in range(args.steps):
            step((args.warmup + i) * nsets)
        torch.cuda.synchronize()
        warm = (time.perf_counter() - w0) * 1e3 / args.steps
    # breakdown pass (not timed): every kernel of at least 50 steps bracketed by events.
    # On short layers the host, at 10-25 us per launch with events, falls behind the
    # device, whose kernels would then start on an idle queue (measured longer than the same
    # kernels behind queued work); a spin of the device (~100 us) queued ahead of each step
    # keeps its kernels behind queued work, as in the timed steps.
    breakdown_steps = max(args.steps, 50)
    ep.trace_reset()
    ep.trace_enable(True)
    for i in range(breakdown_steps):
        if not every:
            torch.cuda._sleep(SPIN_CYCLES)
        step(args.warmup + args.steps + i)
    torch.cuda.synchronize()
    ep.trace_enable(False)
    breakdown = ep.trace_read()
    progress(f"breakdown pass ({breakdown_steps} traced steps) done")
    # graph-replayed steps: one step per buffer set captured once in a HIP graph, replayed;
    # the host then issues one launch per replay instead of two library calls per step
    # (what a decode loop under graph capture does), so layers shorter than the host's
    # issue time show their kernel-bound time
    graph = graph_replayed_steps(step, nsets, max(2, -(-args.steps // nsets)), payload)
    progress("graph-replayed steps done")
    # the roofline's launch averages come from the timed region on long layers (the traced
    # launches of it), from the breakdown pass on short ones; other kernels from the
    # breakdown pass
    kstats = dict(timed_stats)
    for name, st_ in breakdown.items():
        kstats.setdefault(name, st_)
    # the two-kernel path (layout, then pack) on the same steps, for comparison, when the
    # one-kernel dispatch covered this layer (its kernel shows in the trace)
    two = None
    if "layout_pack" in kstats:
        for i in range(args.warmup):
            step(i, fused=False)
        torch.cuda.synchronize()
        u0 = time.perf_counter()
        for i in range(args.steps):
            step(args.warmup + i, fused=False)
        torch.cuda.synchronize()
        two_ms = (time.perf_counter() - u0) * 1e3 / args.steps
        ep.trace_reset()
        ep.trace_enable(True)
        for i in range(args.steps):
            step(args.warmup + args.steps + i, fused=False)
        torch.cuda.synchronize()
        ep.trace_enable(False)
        two = {"note": "the same layer with layout and pack as two calls (two kernels); event-bracketed kernel "
                       "averages",
               "us_per_layer": round(two_ms * 1e3, 2), "payload_GBps": round(2 * payload / (two_ms * 1e-3) / 1e9, 1),
               "kernel_avg_us": {name: round(st_["mean_ms"] * 1e3, 3) for name, st_ in ep.trace_read().items()}}

    abytes = algorithmic_bytes(cfg)
    kernels = {}
    for name, st in kstats.items():
        us = st["mean_ms"] * 1e3
        entry = {"launches": st["count"], "avg_us": round(us, 3),
                 "p10_us": round(st["p10_ms"] * 1e3, 3), "p50_us": round(st["p50_ms"] * 1e3, 3),
                 "p90_us": round(st["p90_ms"] * 1e3, 3),
                 "measured": "timed region, every other step (dispatch and combine alternate)"
                 if name in timed_stats else
                 ("breakdown pass, every launch" if every else
                  "breakdown pass, every launch (the timed steps of layers under 300 us run without events)")}
        if name in abytes and us > 0:
            entry["algorithmic_bytes"] = abytes[name]
            entry["GBps"] = round(abytes[name] / (us * 1e-6) / 1e9, 1)
            entry["hbm_frac"] = round(entry["GBps"] / HBM_PEAK_GBPS, 4)
        kernels[name] = entry
    dominant = max(TIMED_KERNELS, key=lambda nm: kernels.get(nm, {}).get("avg_us", 0.0))
    dk = kernels[dominant]
    traffic = committed_traffic(args.workload, dominant)

    # ---- attainable HBM bandwidth: plain streaming copy of 1 GiB
    a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    for _ in range(2):
        ep.copy_probe(b, a)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(5):
        ep.copy_probe(b, a)
    ev1.record()
    torch.cuda.synchronize()
    copy_gbps = 2 * (1 << 30) * 5 / (ev0.elapsed_time(ev1) * 1e-3) / 1e9
    del a, b
    same_copy = same_bytes_copy(dev, abytes[dominant], nsets)
    ceilings = streaming_ceilings(cfg, dev)
    dest_streams = pack_destination_streams(cfg, staging, [st["x"] for st in sets], nsets, dev)
    progress("copy probes, streaming ceilings and pack destination streams done")

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name} MoE layer: T={T} tokens, H={H}, E={E} experts, top-{k}, "
                        f"R={R}-rank EP group (rank 0 on one GPU), HBM staging",
            "T": T, "H": H, "E": E, "k": k, "R": R, "staging": "hbm",
            "payload_bytes_per_op": payload, "us_per_layer": round(ms_per_step * 1e3, 2),
            "buffer_sets_rotated": nsets, "parallelism": "1 GPU (one EP rank)",
            "host_issue_us_per_step": round(issue_us, 1),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": dominant,
            "achieved": dk.get("GBps"),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": dk.get("hbm_frac"),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": dk.get("algorithmic_bytes"),
            "avg_launch_us": dk.get("avg_us"),
            "p50_launch_us": dk.get("p50_us"),
            "launches_averaged": dk.get("launches"),
            "measured": dk.get("measured"),
            "dispatch_and_combine": pair_roofline(kernels),
            "streaming_ceiling": ceiling_of(dominant, dk.get("hbm_frac"), ceilings, k),
        },
        "kernels": kernels,
        "hbm_copy_probe_GBps": round(copy_gbps, 1),
        "same_bytes_copy": dict(same_copy, kernel=dominant,
                                kernel_speed_vs_copy=round(same_copy["avg_us"] / dk["avg_us"], 3)),
        "streaming_ceilings": ceilings,
        "pack_destination_streams": dest_streams,
    }
    if warm is not None:
        result["warm_cache"] = {
            "note": "the same steps on one buffer set: inputs and staging stay in the memory-side cache "
                    "(the headline rotates sets so that they do not)",
            "us_per_layer": round(warm * 1e3, 2),
            "payload_GBps": round(2 * payload / (warm * 1e-3) / 1e9, 1),
        }
    if two is not None:
        result["two_kernel_dispatch"] = two
    result["graph_replayed_steps"] = graph

    # ---- pinned host staging: the same layer with SDMA legs, host flags, simulated peers
    if not args.no_pinned:
        result["pinned_staging"] = bench_pinned(cfg, inp, y, args, dev)
        progress("pinned staging done")

    # ---- CPU baseline: the oracle on whole layers of the same workload, on all the host
    #      cores this process may use, and on one
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(cfg, inp, y, args.cpu_seconds)
        progress("CPU baseline done")

    print(json.dumps(result))


PINNED_MODES = (
    # name, mode bits (EP_MODE_*: 1 per-sender, 2 duplex, 4 remote-only, 8 accumulate as senders land)
    ("default", 0),
    ("per_sender", 1),
    ("duplex", 2),
    ("duplex_per_sender", 3),
    ("duplex_remote_only_per_sender", 7),
    ("per_sender_accumulate", 9),
    ("duplex_per_sender_accumulate", 11),
)


def graph_replayed_steps(step, nsets: int, replays: int, payload: int) -> dict:
    """The layer's steps (one per buffer set, the timed region's rotation) captured in one
    HIP graph and replayed `replays` times; us per layer from the host clock around the
    replays."""
    import torch
    try:
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cs):
            with torch.cuda.graph(g, stream=cs):
                for i in range(nsets):
                    step(i)
        torch.cuda.current_stream().wait_stream(cs)
        for _ in range(2):
            g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(replays):
            g.replay()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / (replays * nsets)
        del g
    except RuntimeError as e:
        return {"error": str(e)}
    return {"us_per_layer": round(ms * 1e3, 2), "payload_GBps": round(2 * payload / (ms * 1e-3) / 1e9, 1),
            "steps": replays * nsets,
            "note": "the same steps (one-kernel dispatch or layout and pack, then combine) captured once per "
                    "buffer set in a HIP graph and replayed: one host launch per replay"}


def pinned_legs(st, x, lay, w, out, k, leg_bytes, peaks, calls, epoch0) -> dict:
    """Rates of the default mode's two host legs, each from back-to-back untraced calls of
    the call that holds it (no simulated peers: the dispatch waits only for its own
    device->host flags, and the combine finds its senders' flags already raised)."""
    import torch

    import paper_2609_40093_amd as ep

    nbuf = st.num_buffers

    def timed(fn):
        for i in range(3):
            fn(i)
        st.status()
        t0 = time.perf_counter()
        for i in range(calls):
            fn(3 + i)
        st.status()
        return (time.perf_counter() - t0) * 1e6 / calls

    d_us = timed(lambda i: ep.dispatch(x, lay.slot_pos, st, topk=k, buf=i % nbuf, epoch=epoch0 + i))
    ready = epoch0 + calls + 100
    for b in range(nbuf):
        st.host_array("recv_flags", b)[:] = ready
    c_us = timed(lambda i: ep.combine(st, lay.slot_pos, w, out=out, buf=i % nbuf, epoch=ready))
    torch.cuda.synchronize()
    res = {}
    for leg, us, peak in (("d2h_leg", d_us, peaks["d2h_alone"]), ("h2d_leg", c_us, peaks["h2d_alone"])):
        gbps = leg_bytes / (us * 1e-6) / 1e9
        res[leg] = {"call_us": round(us, 1), "bytes": leg_bytes, "GBps_lower_bound": round(gbps, 2),
                    "frac_of_measured_peak_lower_bound": round(gbps / peak, 3)}
    return res


def staging_flags(st) -> dict:
    """Every host flag word of a pinned staging, per buffer set (reported with a failed mode)."""
    import ctypes

    def words(ptr, n):
        return list((ctypes.c_uint32 * n).from_address(ptr)) if ptr and n > 0 else None
    out = {}
    for b, v in enumerate(st.views):
        R = v.num_ranks
        out[str(b)] = {"mode": v.mode, "send": words(v.send_flags, v.max_chunks), "recv": words(v.recv_flags, R),
                       "in": words(v.in_flags, R), "ret": words(v.ret_flags, R), "in_landed": words(v.in_landed, R),
                       "recv_landed": words(v.recv_landed, R)}
    return out


def bench_pinned(cfg, inp, y, args, dev) -> dict:
    """The same layer with pinned host staging, in each exchange mode.  Simulated peers
    announce their rows at once (no skew).  In the duplex modes every sender r sends this
    rank as many rows as it sends r (a symmetric traffic matrix), so each phase moves the
    same bytes both ways; PCIe bytes per layer count both directions."""
    import numpy as np
    import torch

    import paper_2609_40093_amd as ep

    T, H, E, k, R = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R
    n = cfg.slots
    rb = 2 * H
    nbuf = 2
    x = torch.from_numpy(inp.x.view(np.int16)).to(dev)
    idx = torch.from_numpy(inp.topk_idx).to(dev)
    w = torch.from_numpy(inp.topk_w).to(dev)
    out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
    lay = ep.dispatch_layout(idx, E, R)
    counts = lay.rank_counts.cpu().numpy().astype(np.int64)
    me = 0
    steps = max(5, min(args.steps // 2, 50))
    peaks = pcie_peaks(dev)
    modes = {}
    for name, mode in PINNED_MODES:
        st = ep.Staging("pinned", n, H, R, num_buffers=nbuf, chunk_bytes=args.chunk_mib << 20)
        if mode:
            st.set_mode(mode, self_rank=me)
        inbound_rows = 0
        for b in range(nbuf):
            st.host_array("recv", b)[:n] = y
            if mode & ep.MODE_DUPLEX:
                rin = counts.copy()
                rin[me] = 0
                st.set_inbound(b, rin)
                inbound_rows = int(rin.sum()) + int(counts[me])
                st.host_array("in", b)[:inbound_rows] = y[:inbound_rows]
        peers = ep.SimPeers(st, echo=False)
        try:

            def step(i):
                buf, epoch = i % nbuf, i + 1
                ep.dispatch_layout(idx, E, R, out=lay)
                peers.post(buf, epoch, n)
                ep.dispatch(x, lay.slot_pos, st, topk=k, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)
                ep.combine(st, lay.slot_pos, w, out=out, buf=buf, epoch=epoch, rank_offsets=lay.rank_offsets)

            for i in range(args.warmup):
                step(i)
            st.status()
            peers.drain()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(steps):
                step(args.warmup + i)
            st.status()
            t1 = time.perf_counter()
            peers.drain()
            ms = (t1 - t0) * 1e3 / steps
            legs = {}
            if mode == 0:
                legs = pinned_legs(st, x, lay, w, out, k, n * rb, peaks, steps, args.warmup + steps)
                # breakdown pass (not timed): the kernels, each bracketed by its launch events
                ep.trace_reset()
                ep.trace_enable(True)
                for i in range(steps):  # epochs above the flags pinned_legs raised
                    step(args.warmup + 3 * steps + 200 + i)
                st.status()
                peers.drain()
                ep.trace_enable(False)
                ks = ep.trace_read()
                legs["kernels_avg_us"] = {kn: round(ks[kn]["mean_ms"] * 1e3, 2) for kn in
                                          ("wait_d2h", "wait_recv", "release_signal", "pack", "combine", "layout")
                                          if kn in ks}
        except ep.EPError as e:
            # a failed mode is reported with its flag words, and the others still run
            modes[name] = {"mode_bits": mode, "error": str(e), "flags": staging_flags(st)}
            peers.close()
            st.close()
            continue
        peers.close()
        st.close()
        progress(f"pinned mode {name}: {ms * 1e3:.0f} us per layer")
        self_rows = int(counts[me]) if mode & ep.MODE_REMOTE_ONLY else 0
        if mode & ep.MODE_DUPLEX:
            pcie = 2 * (n - self_rows) * rb + 2 * (inbound_rows - self_rows) * rb
            peak = peaks["both"]
            # dispatch: this rank's rows up, the inbound rows down; combine: the results for
            # the other senders up, the returned rows down
            phases = [((n - self_rows) * rb, (inbound_rows - self_rows) * rb),
                      ((inbound_rows - self_rows) * rb, (n - self_rows) * rb)]
        else:
            pcie = 2 * n * rb
            peak = peaks["d2h_alone"]
            phases = [(n * rb, 0), (0, n * rb)]
        bound_us = pattern_bound_us(phases, peaks)
        gbps = pcie / (ms * 1e-3) / 1e9
        modes[name] = {
            "mode_bits": mode,
            "us_per_layer": round(ms * 1e3, 1),
            "payload_GBps": round(2 * cfg.payload_bytes / (ms * 1e-3) / 1e9, 2),
            "pcie_bytes_per_layer": pcie,
            "pcie_GBps": round(gbps, 2),
            "pcie_peak_used_GBps": peak,
            "frac_of_measured_pcie_peak": round(gbps / peak, 3),
            "pcie_pattern_bound_us": round(bound_us, 1),
            "frac_of_pattern_bound": round(bound_us / (ms * 1e3), 3),
        }
        if legs:
            modes[name]["legs"] = legs
            modes[name]["legs_note"] = ("each host leg timed as back-to-back untraced calls of its call alone "
                                        "(dispatch: pack + device->host leg + flag wait; combine: flag wait with the "
                                        "flags already up + host->device leg + reduction), so each rate is a lower "
                                        "bound on the leg's own; kernel times from a separate traced pass")

    def section(fn, *a):  # a failed section is reported, and the others still run
        try:
            return fn(*a)
        except ep.EPError as e:
            return {"error": str(e)}
    dense = section(bench_dense, cfg, inp, args, dev, peaks)
    progress("dense All-Gather / Reduce-Scatter layer done")
    graph = section(bench_graph, ["decode", cfg.name], args, dev, peaks)
    progress("graph-replayed rounds done")
    decode_latency = section(bench_decode_latency, args, dev)
    return {
        "decode_dispatch_host_latency": decode_latency,
        "graph_replayed_rounds": graph,
        "steps": steps,
        "chunk_bytes": args.chunk_mib << 20,
        "modes": modes,
        "dense_allgather_reducescatter": dense,
        "pcie_measured_peak_GBps": peaks,
        "pcie_published_peak_GBps": PCIE_PEAK_GBPS,
        "note": "default and per_sender move T*k rows each way per layer (one direction per phase); "
                "the duplex modes also move the rows other senders dispatch to this rank and this rank's "
                "results for them (symmetric traffic), so each phase uses both PCIe directions; the "
                "duplex peak is the two-engine bidirectional probe",
    }


def bench_decode_latency(args, dev, rounds: int = 60) -> dict:
    """Decode-shaped layer (T = 256, H = 7168, top-8 of 256, R = 8), pinned staging, default
    mode: time from enqueueing the dispatch (layout, pack, SDMA leg) until a host thread sees
    the last chunk's completion flag in host memory, one round at a time."""
    import numpy as np
    import torch

    import paper_2609_40093_amd as ep
    from paper_2609_40093_amd import synth

    cfg = synth.config("decode")
    inp = synth.make_inputs(cfg)
    T, H, E, k, R = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R
    n = cfg.slots
    st = ep.Staging("pinned", n, H, R, num_buffers=2)   # default chunk: the layer is one chunk
    x = torch.from_numpy(inp.x.view(np.int16)).to(dev)
    idx = torch.from_numpy(inp.topk_idx).to(dev)
    last = (n * 2 * H + st.chunk_bytes - 1) // st.chunk_bytes - 1
    lay = None
    lat = []
    for i in range(args.warmup + rounds):
        buf, epoch = i % 2, i + 1
        flags = st.host_array("send_flags", buf)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        lay = ep.dispatch_fused(x, idx, E, R, st, buf=buf, epoch=epoch, out=lay)
        while int(flags[last]) != epoch:
            if time.perf_counter() - t0 > 5.0:
                raise RuntimeError("decode dispatch flag did not arrive within 5 s")
        t1 = time.perf_counter()
        torch.cuda.synchronize()
        if i >= args.warmup:
            lat.append((t1 - t0) * 1e6)
    st.status()
    ep.layout_validate(lay)
    st.close()
    lat = np.array(lat)
    return {
        "workload": f"decode layer: T={T}, H={H}, top-{k} of {E}, R={R}, pinned staging, default mode",
        "bytes": n * 2 * H,
        "us_p10": round(float(np.percentile(lat, 10)), 1),
        "us_p50": round(float(np.percentile(lat, 50)), 1),
        "us_p90": round(float(np.percentile(lat, 90)), 1),
        "rounds": rounds,
        "note": "host-observed: enqueue of layout + pack + SDMA leg until a host thread polling host memory "
                "sees the last chunk's flag; includes the host's launch calls",
    }


def bench_dense(cfg, inp, args, dev, peaks) -> dict:
    """The paper's adopted design for the same layer (Sec. 4.2): single-step All-Gather of
    every rank's T tokens, grouping of the R*T gathered tokens by this rank's experts,
    identity experts, partial blocks (bf16), Reduce-Scatter with GPU or partial host
    reduction.  The other ranks' shards and blocks are seeded data their simulated peers
    announce at once; their routing is this rank's routing rotated over the tokens (the
    same distribution)."""
    import numpy as np
    import torch

    import paper_2609_40093_amd as ep
    from paper_2609_40093_amd import synth

    T, H, E, k, R = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R
    me, L, nbuf = 0, cfg.E // cfg.R, 2
    idx_all = np.concatenate([np.roll(inp.topk_idx, r * T // R, axis=0) for r in range(R)])
    w_all = np.concatenate([np.roll(inp.topk_w, r * T // R, axis=0) for r in range(R)])
    idx_d = torch.from_numpy(idx_all).to(dev)
    w_d = torch.from_numpy(w_all).to(dev)
    x = torch.from_numpy(inp.x.view(np.int16)).to(dev)
    res = {}
    for name, on_host in (("gpu_reduction", False), ("partial_host_reduction", True)):
        d = ep.Dense(T, H, R, self_rank=me, num_buffers=nbuf)
        d.set_policy(per_sender=True)
        for b in range(nbuf):
            hag, hin = d.host_array("ag", b), d.host_array("rs_in", b)
            for r in range(R):
                if r != me:
                    rows = synth.normal_bf16_rows(np.random.SeedSequence([cfg.seed, 7, r]), T, H)
                    hag[r * T:(r + 1) * T] = rows
                    hin[r * T:(r + 1) * T] = rows
        peers = ep.SimPeers(d)
        lay = ep.dispatch_layout_local(idx_d, E, me * L, (me + 1) * L)
        y_local = torch.empty((R * T * k, H), dtype=torch.int16, device=dev)   # every local row fits
        blocks = torch.empty((R * T, H), dtype=torch.bfloat16, device=dev)
        out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)

        def step(i):
            buf, epoch = i % nbuf, i + 1
            peers.post_dense(buf, epoch, "ag")
            ep.allgather(d, x, buf=buf, epoch=epoch)
            ep.dispatch_layout_local(idx_d, E, me * L, (me + 1) * L, out=lay)
            g = d.views[buf].dev_gathered
            # pack straight from the gathered device buffer (raw pointer of the staging)
            ep.api._check(ep.api._lib_handle().ep_pack(ctypes.c_void_p(g), R * T, H, k, ep.api._ptr(lay.slot_pos),
                                                       ep.api._ptr(y_local), y_local.shape[0],
                                                       ep.api._stream_ptr(None)), "ep_pack")
            ep.combine_rows(y_local, lay.slot_pos, w_d, blocks)
            peers.post_dense(buf, epoch, "rs")
            ep.reducescatter(d, blocks, num_tokens=T, out=out, reduce_on_host=on_host, buf=buf, epoch=epoch)

        steps = max(5, min(args.steps // 4, 25))
        for i in range(args.warmup):
            step(i)
        d.status()
        peers.drain()
        up0, down0 = d.bytes_moved()
        t0 = time.perf_counter()
        for i in range(steps):
            step(args.warmup + i)
        d.status()
        t1 = time.perf_counter()
        up1, down1 = d.bytes_moved()
        peers.drain()
        # breakdown pass (not timed): kernels, gates and the host reduction
        ep.trace_reset()
        ep.trace_enable(True)
        for i in range(steps):
            step(args.warmup + steps + i)
        d.status()
        peers.drain()
        ep.trace_enable(False)
        ks = ep.trace_read()
        peers.close()
        d.close()
        ms = (t1 - t0) * 1e3 / steps
        pcie = ((up1 - up0) + (down1 - down0)) / steps
        gbps = pcie / (ms * 1e-3) / 1e9
        S = T * H * 2
        # All-Gather: S up, (R-1)S down; Reduce-Scatter: (R-1)S up, (R-1)S or S down
        phases = [(S, (R - 1) * S), ((R - 1) * S, S if on_host else (R - 1) * S)]
        bound_us = pattern_bound_us(phases, peaks)
        res[name] = {"us_per_layer": round(ms * 1e3, 1), "pcie_bytes_per_layer": int(pcie),
                     "pcie_up_down_per_layer": [int((up1 - up0) / steps), int((down1 - down0) / steps)],
                     "pcie_GBps": round(gbps, 2), "frac_of_measured_pcie_peak": round(gbps / peaks["both"], 3),
                     "pcie_pattern_bound_us": round(bound_us, 1),
                     "frac_of_pattern_bound": round(bound_us / (ms * 1e3), 3),
                     "breakdown_avg_us": {kn: round(v["mean_ms"] * 1e3, 1) for kn, v in ks.items()}}
    res["note"] = ("per-sender policy; payload per layer: All-Gather S up + (R-1)S down, Reduce-Scatter (R-1)S up "
                   "and (R-1)S down (GPU reduction) or S down (host reduction), S = T*H*2 bytes")
    return res


def bench_graph(names, args, dev, peaks) -> dict:
    """Graph-replayed rounds (the decode path, Sec. 4.5): one round -- round counter,
    layout, dispatch, combine -- captured once in a HIP graph and replayed back to back,
    with each of the two kinds of host legs: the compute units storing the rows to and
    loading them from pinned memory (`compute_unit_legs`), or SDMA engines driven by the
    library's host-leg thread, the captured kernels packing into and reducing from device
    memory (`sdma_legs`, ep_graph_legs_sdma).  The simulated peers only raise flags and
    credits (their returned rows are seeded data already in the pinned receive buffers)."""
    import numpy as np
    import torch

    import paper_2609_40093_amd as ep
    from paper_2609_40093_amd import synth

    res = {}
    for name in names:
        cfg = synth.config(name)
        inp = synth.make_inputs(cfg)
        T, H, E, k, R, n = cfg.T, cfg.H, cfg.E, cfg.k, cfg.R, cfg.slots
        y = inp.expert_outputs()
        x = torch.from_numpy(inp.x.view(np.int16)).to(dev)
        idx = torch.from_numpy(inp.topk_idx).to(dev)
        w = torch.from_numpy(inp.topk_w).to(dev)
        out = torch.empty((T, H), dtype=torch.bfloat16, device=dev)
        res[name] = {}
        for legs in ("compute_unit_legs", "sdma_legs"):
            st = ep.Staging("pinned", n, H, R, num_buffers=2)
            for b in range(2):
                st.host_array("recv", b)[:n] = y
            peers = ep.SimPeers(st, echo=False, graph_rows=n)
            if legs == "sdma_legs":
                ep.graph_legs_sdma(st, True)
            lay = ep.dispatch_layout(idx, E, R)
            unsettled = settle_h2d(dev)

            def one_round():
                ep.round_advance(st)
                ep.dispatch_layout(idx, E, R, out=lay)
                ep.dispatch_graph(x, lay.slot_pos, st, topk=k)
                ep.combine_graph(st, lay.slot_pos, w, out)

            one_round()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                with torch.cuda.graph(g, stream=s):
                    one_round()
            torch.cuda.current_stream().wait_stream(s)
            for _ in range(args.warmup):
                g.replay()
            torch.cuda.synchronize()
            steps = max(10, min(args.steps, 100))
            t0 = time.perf_counter()
            for _ in range(steps):
                g.replay()
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            st.status()
            rounds = ep.round_read(st)
            peers.wait_round(rounds)
            peers.close()
            del g
            st.close()
            us = (t1 - t0) * 1e6 / steps
            pcie = 2 * n * 2 * H
            gbps = pcie / (us * 1e-6) / 1e9
            res[name][legs] = {"us_per_round": round(us, 1), "pcie_bytes_per_round": pcie,
                               "pcie_GBps": round(gbps, 2),
                               "frac_of_one_way_pcie_peak": round(gbps / peaks["d2h_alone"], 3), "replays": steps}
            if unsettled:
                res[name][legs]["earlier_unsettled_probes"] = unsettled
    res["note"] = ("compute_unit_legs: rows stored to and loaded from pinned memory by the compute units; sdma_legs: "
                   "rows packed into and reduced from device memory by the captured kernels and moved by SDMA "
                   "engines (the library's host-leg thread); the two directions run one after the other within a "
                   "round, so the one-way peak bounds the rate; each measurement starts once host->device copies "
                   "run within 20% of device->host ones (settle_h2d)")
    return res


def pattern_bound_us(phases, peaks) -> float:
    """The least time the PCIe traffic of a layer can take at the measured peaks: phase by
    phase (each a list of (bytes up, bytes down) moving at once), the largest of the
    upload at the one-way device->host peak, the download at the one-way host->device peak
    and both together at the two-way peak."""
    t = 0.0
    for up, down in phases:
        t += max(up / peaks["d2h_alone"], down / peaks["h2d_alone"], (up + down) / peaks["both"]) / 1e3
    return t


def pcie_peaks(dev) -> dict:
    """SDMA copies of 1 GiB between pinned host memory and HBM on the exchange's engines
    (ep_pcie_probe, best of four timed runs): each direction alone and both at once on two
    engines, on two separately allocated pinned buffers, the faster of the two per
    direction."""
    import torch

    import paper_2609_40093_amd as ep
    nbytes = 1 << 30
    hosts = [torch.empty(2 * nbytes, dtype=torch.uint8, pin_memory=True) for _ in range(2)]
    devb = torch.empty(2 * nbytes, dtype=torch.uint8, device=dev)

    def probe():
        runs = []
        for host in hosts:
            runs.append({"d2h_alone": round(ep.pcie_probe(host, devb, nbytes, 1), 2),
                         "h2d_alone": round(ep.pcie_probe(host, devb, nbytes, 2), 2),
                         "both": round(ep.pcie_probe(host, devb, nbytes, 3), 2)})
        return runs
    # Both one-way rates are about 57 GB/s on this machine.  For a few seconds after a
    # process that held tens of GB of pinned memory has exited, host->device copies run at
    # about half that, on every buffer; the section waits (up to 10 s) until the two one-way
    # rates agree within 20% before it measures anything.
    runs = probe()
    unsettled = []
    deadline = time.perf_counter() + 10.0
    while (max(r["h2d_alone"] for r in runs) < 0.8 * max(r["d2h_alone"] for r in runs)
           and time.perf_counter() < deadline):
        unsettled.append(runs)
        time.sleep(1.0)
        runs = probe()
    del hosts, devb
    res = {key: max(r[key] for r in runs) for key in runs[0]}
    res["per_buffer"] = runs
    if unsettled:
        res["earlier_unsettled_probes"] = unsettled
    return res


def settle_h2d(dev, max_s: float = 10.0) -> list:
    """Waits (up to max_s) until host->device SDMA copies run within 20% of device->host
    ones (256 MiB probes on one pinned buffer): after a process, or an earlier section,
    freed tens of GB of pinned memory, host->device copies run at about half their rate
    for a few seconds.  Returns the probes taken while they had not settled."""
    import torch

    import paper_2609_40093_amd as ep
    nbytes = 256 << 20
    host = torch.empty(2 * nbytes, dtype=torch.uint8, pin_memory=True)
    devb = torch.empty(2 * nbytes, dtype=torch.uint8, device=dev)
    unsettled = []
    deadline = time.perf_counter() + max_s
    while True:
        d2h, h2d = ep.pcie_probe(host, devb, nbytes, 1), ep.pcie_probe(host, devb, nbytes, 2)
        if h2d >= 0.8 * d2h or time.perf_counter() >= deadline:
            break
        unsettled.append({"d2h_alone": round(d2h, 2), "h2d_alone": round(h2d, 2)})
        time.sleep(0.5)
    del host, devb
    return unsettled


def ceiling_of(kernel: str, frac, ceilings: dict, k: int) -> dict:
    """What plain streaming code reaches for the kernel's traffic (the fastest store policy):
    the write-only stream for the dispatch kernels (89% or more of their bytes are writes at
    top-8, 67% at top-2), the k:1 stream for the combine."""
    base = f"combine_like_{k}_to_1" if kernel == "combine" else "write_only"
    names = [base, base + "_write_through", base + "_write_through_nt"]
    got = [(ceilings[n]["frac"], n) for n in names if isinstance(ceilings.get(n), dict)]
    if not got or not frac:
        return {"note": "no streaming probe at this row size"}
    best, name = max(got)
    return {"mix": name, "frac": best, "kernel_frac_of_ceiling": round(frac / best, 3)}


def pair_roofline(kernels: dict) -> dict:
    """The dispatch kernel and combine of one layer together: their algorithmic bytes over
    their summed average durations, against the HBM peak."""
    disp = "layout_pack" if "layout_pack" in kernels else "pack"
    pair = [kernels[disp], kernels["combine"]]
    nbytes = sum(k["algorithmic_bytes"] for k in pair)
    us = sum(k["avg_us"] for k in pair)
    gbps = nbytes / (us * 1e-6) / 1e9
    return {"kernels": [disp, "combine"], "algorithmic_bytes": nbytes, "avg_us": round(us, 3),
            "achieved": round(gbps, 1), "frac": round(gbps / HBM_PEAK_GBPS, 4)}


def same_bytes_copy(dev, nbytes: int, nsets: int, launches: int = 40) -> dict:
    """The library's plain streaming copy moving `nbytes` per launch (half read, half
    written), over `nsets` rotated buffer pairs and timed by the same launch events as the
    path's kernels: what simple streaming code reaches on this chip at this size."""
    import torch

    import paper_2609_40093_amd as ep
    half = nbytes // 2 // 4096 * 4096
    pairs = [(torch.empty(half, dtype=torch.uint8, device=dev), torch.empty(half, dtype=torch.uint8, device=dev))
             for _ in range(nsets)]
    for j in range(2 * nsets):
        ep.copy_probe(pairs[j % nsets][1], pairs[j % nsets][0])
    torch.cuda.synchronize()
    ep.trace_reset()
    ep.trace_enable(True)
    for j in range(launches):
        ep.copy_probe(pairs[j % nsets][1], pairs[j % nsets][0])
    torch.cuda.synchronize()
    ep.trace_enable(False)
    st = ep.trace_read()["copy_probe"]
    ep.trace_reset()
    us = st["mean_ms"] * 1e3
    return {"bytes_per_launch": 2 * half, "launches": st["count"], "avg_us": round(us, 3),
            "p50_us": round(st["p50_ms"] * 1e3, 3), "GBps": round(2 * half / (us * 1e-6) / 1e9, 1)}


def streaming_ceilings(cfg, dev, launches: int = 10) -> dict:
    """What plain streaming code attains at this layer's size (ep_stream_probe): every mix
    moves the rows of one dispatch, (k+1)*T rows of 2H bytes, over sequential addresses --
    1 read : k writes like the pack, k reads : 1 write like the combine, copy 1:1,
    read-only and write-only -- on buffer sets rotated past the memory-side cache, each
    launch timed by events.  Fractions are of the 8 TB/s peak."""
    import torch

    import paper_2609_40093_amd as ep
    T, H, k = cfg.T, cfg.H, cfg.k
    row = 2 * H
    if row % 1024 or row // 1024 not in (1, 2, 4, 8, 14, 16):
        return {"note": f"rows of {row} bytes: no probe instance"}
    rows = (k + 1) * T
    set_bytes = rows * row
    nsets = max(1, min(8, -(-3 * MALL_BYTES // set_bytes)))
    src = torch.empty(nsets * set_bytes, dtype=torch.uint8, device=dev)
    dst = torch.empty(nsets * set_bytes, dtype=torch.uint8, device=dev)
    src.fill_(1)
    mixes = {f"pack_like_1_to_{k}": (T, 1, k), f"combine_like_{k}_to_1": (T, k, 1),
             "copy_1_to_1": (rows // 2, 1, 1), "read_only": (rows, 1, 0), "write_only": (rows, 0, 1)}
    runs = []
    for name, (units, r, w) in mixes.items():
        runs.append((name, units, r, w, 0))
        if w:  # the same mix with the path's other store policies
            runs += [(name + "_write_through", units, r, w, 1), (name + "_write_through_nt", units, r, w, 2)]
    res = {}
    for name, units, r, w, pol in runs:
        def launch(j):
            off = (j % nsets) * set_bytes
            ep.stream_probe(dst[off:], src[off:], units, row, r, w, store_policy=pol)
        for j in range(2):
            launch(j)
        torch.cuda.synchronize()
        ep.trace_reset()
        ep.trace_enable(True)
        for j in range(launches):
            launch(j)
        torch.cuda.synchronize()
        ep.trace_enable(False)
        st = ep.trace_read()["stream_probe"]
        ep.trace_reset()
        us = st["mean_ms"] * 1e3
        nbytes = units * (r + w) * row
        gbps = nbytes / (us * 1e-6) / 1e9
        res[name] = {"units": units, "reads": r, "writes": w, "row_bytes": row, "bytes_per_launch": nbytes,
                     "launches": st["count"], "avg_us": round(us, 2), "GBps": round(gbps, 1),
                     "frac": round(gbps / HBM_PEAK_GBPS, 4)}
    del src, dst
    res["note"] = ("ep_stream_probe over sequential addresses, 16-byte vectors, one wave per unit, non-temporal "
                   "stores (names ending _write_through: device-scope write-through buffer stores; _write_through_nt: "
                   "the same with the non-temporal hint); buffer sets rotated "
                   "past the 256 MB memory-side cache")
    return res


def pack_destination_streams(cfg, staging, xs, nsets: int, dev, launches: int = 6) -> dict:
    """The path's own pack (ep_dispatch on HBM staging) with synthetic routings whose rows go
    to S destination regions, each entry to a region drawn uniformly and rows grouped
    stably by region as the layout groups them by expert -- S = 1 is the identity (each
    token's k rows side by side), S = E the uniform routing over the layer's experts.  The
    pack's bytes do not change with S; its time shows what HBM gives for S concurrent
    write streams.  Launches rotate over the layer's buffer sets and are timed by events."""
    import numpy as np
    import torch

    import paper_2609_40093_amd as ep
    T, H, k, E = cfg.T, cfg.H, cfg.k, cfg.E
    n = T * k
    nbytes = T * 2 * H + n * 2 * H + 4 * n
    rng = np.random.default_rng(20260601)
    res = {}
    for S in sorted({1, 8, 32, E}):
        if S == 1:
            pos = np.arange(n, dtype=np.int32)
        else:
            region = rng.integers(0, S, size=n)
            pos = np.empty(n, dtype=np.int32)
            pos[np.argsort(region, kind="stable")] = np.arange(n, dtype=np.int32)
        sp = torch.from_numpy(pos).to(dev)
        for j in range(2):
            ep.dispatch(xs[j % len(xs)], sp, staging, topk=k, buf=j % nsets, epoch=1)
        torch.cuda.synchronize()
        ep.trace_reset()
        ep.trace_enable(True)
        for j in range(launches):
            ep.dispatch(xs[j % len(xs)], sp, staging, topk=k, buf=j % nsets, epoch=1)
        torch.cuda.synchronize()
        ep.trace_enable(False)
        st = ep.trace_read()["pack"]
        ep.trace_reset()
        us = st["mean_ms"] * 1e3
        gbps = nbytes / (us * 1e-6) / 1e9
        res[f"streams_{S}"] = {"launches": st["count"], "avg_us": round(us, 2), "GBps": round(gbps, 1),
                               "frac": round(gbps / HBM_PEAK_GBPS, 4)}
        del sp
    res["note"] = ("ep_dispatch's pack on synthetic routings to S regions (uniform); the layer's own routing "
                   "is skewed over its experts and sits between these figures")
    return res


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, inp, y, seconds: float) -> dict:
    """The oracle as it stands (plain C, fp64 sums) over whole layers of the workload: its
    layout, pack and combine, on every host core this process may use (the oracle's token
    loops split over threads, outputs identical to one thread's), and on one thread.  The
    output arrays are allocated and touched once before the clock starts, so that the
    figure is the oracle's work and not the host's first-touch page faults; each figure
    runs whole layers until `seconds` have passed (at least one)."""
    import numpy as np

    import oracle
    lib = oracle.load()
    T, H, k = cfg.T, cfg.H, cfg.k
    x = np.ascontiguousarray(inp.x)
    w = np.ascontiguousarray(inp.topk_w)
    y = np.ascontiguousarray(y)
    packed = np.empty((max(T * k, 1), H), np.uint16)
    exact = np.empty((max(T, 1), H), np.float64)
    b16 = np.empty((max(T, 1), H), np.uint16)
    f32 = np.empty((max(T, 1), H), np.float32)
    for a in (packed, exact, b16, f32):
        a.fill(0)

    def layers(threads: int):
        oracle.set_threads(threads)
        passes, t0 = 0, time.perf_counter()
        try:
            while True:
                lay = oracle.layout(inp.topk_idx, cfg.E, cfg.R, lib=lib)
                sp = np.ascontiguousarray(lay.slot_pos)
                lib.ep_oracle_pack(x, T, H, k, sp, packed)
                lib.ep_oracle_combine(y, sp, w, T, H, k, exact.ctypes.data, b16.ctypes.data, f32.ctypes.data)
                passes += 1
                el = time.perf_counter() - t0
                if el >= seconds:
                    return passes, el
        finally:
            oracle.set_threads(1)

    cores = len(os.sched_getaffinity(0))
    res = {}
    for name, threads in (("all_cores", cores), ("single_thread", 1)):
        passes, el = layers(threads)
        res[name] = {"value": round(2 * cfg.payload_bytes * passes / el / 1e9, 4), "unit": "GB/s",
                     "cores": threads, "us_per_layer": round(el / passes * 1e6, 1),
                     "sample": f"{passes} whole {cfg.name} layer(s) (layout + pack + combine with fp64 sums), "
                               f"{el:.1f} s on {threads} host thread(s)"}
    top = dict(res["all_cores"])
    top.update(kind="oracle", cpu_model=cpu_model(), cores_available=cores,
               single_thread=res["single_thread"],
               note="the oracle's token loops of pack and combine split over threads (OpenMP); its layout's "
                    "counting pass runs on one thread; outputs identical for any thread count")
    return top


if __name__ == "__main__":
    main()
