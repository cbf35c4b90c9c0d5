#!/usr/bin/env python3
"""Benchmark of the band-attention hot path on one MI355X.

One step = sa_forward + sa_backward over one batch of the SA forward+backward
workload (B=16, T=800, H=12, d=64, Lb=64, La=8, lengths U[400, 800], bf16,
synthetic N(0,1)/sqrt(d) inputs and N(0,1) upstream gradient). The headline
value is valid frames per second over the whole step. Inputs are resident in
HBM before timing; four copies of the batch are rotated so that no step finds
its inputs in the 256 MB Infinity Cache. Every timed loop starts after 50 ms
of the same launches back to back (``clock_ramp_ms``), so that it measures the
kernels at the GPU's working clocks rather than their ramp from idle; the W
warmup steps follow the ramp.

The same run also measures:
  * the device-copy reference of the library at the backward's traffic size,
    the practical bandwidth ceiling (row "copy_ceiling"; the roofline object
    carries it and the achieved fraction of it);
  * sa_forward at the paper's l32_r8 window, B=8, T=500 (row
    "sa_forward_l32_r8");
  * llsa_forward and llsa_backward, two-branch, same shapes (rows "llsa",
    "llsa_backward");
  * llsa_paper_forward and llsa_paper_backward, the paper's channel form with
    La + 1 = 9 channels, same shapes (rows "llsa_paper",
    "llsa_paper_backward");
  * sa_stream_step, 64 streams x 1000 steps, ring of 64 + 8 + 1 frames, eager
    and replayed from a HIP graph (row "stream"), and llsa_stream_step on the
    same shapes (row "llsa_stream"), each against the launch floor (an empty
    launch, eager and from a graph), which bounds them;
  * the algorithmic latency of a 12-layer streaming stack, SA against LLSA
    (row "stream_latency");
  * masked full attention in PyTorch (dense T x T scores, band mask) as the
    GPU baseline the paper argues against, and torch's
    scaled_dot_product_attention with a boolean band mask (row
    "masked_attention_torch");
  * the CPU oracle on every host core the process may use, on one core, and
    on the other configurations (``cpu_baseline``).

Prints one JSON line. ``--gpus N`` with N > 1 is not supported (one GPU).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2302_13451_amd import accounting as acc  # noqa: E402
from paper_2302_13451_amd import binding as bd  # noqa: E402
from paper_2302_13451_amd.inputs import llsa_inputs, sa_inputs, stream_inputs  # noqa: E402

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, published
BF16_DENSE_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, published

WORKLOAD = dict(B=16, T=800, H=12, d=64, Lb=64, La=8, lengths=(400, 800), seed=3)
STREAM = dict(S=64, H=12, d=64, Lb=64, La=8, steps=1000, seed=5)
N_SETS = 4
# Seconds of back-to-back launches of the same calls before every timed loop:
# from idle the GPU takes some tens of milliseconds of sustained load to reach
# its working clocks, and a loop timed before that (the headline step at 5
# warmup steps reads about 58 us instead of 54 us) measures the ramp, not the
# kernels. The W warmup steps of the contract follow the ramp.
RAMP_S = 0.05


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def source_sha(*names):
    """Hash of the kernel sources a counter summary was taken on (the shared
    device header included)."""
    h = hashlib.sha256()
    for n in names + ("device_common.h",):
        with open(os.path.join(ROOT, "paper_2302_13451_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_mfma(profile_name, sha):
    """MFMA rate of the kernel from the committed rocprofv3 SQ-counter summary
    (bf16 MFMA operations per launch over the kernel's duration, against the
    dense bf16 peak), if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", profile_name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha") != sha:
        return None
    return {k: rec.get(k) for k in ("mfma_tflops", "mfma_frac_of_bf16_peak", "valu_busy",
                                    "lds_bank_conflict_frac", "mfma_busy")}


def load_traffic(profile_name, sha):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", profile_name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha") != sha:
        return None
    return rec.get("traffic_bytes_per_launch")


class EventTimer:
    """Accumulates the duration of one kernel launch at a time with HIP events
    recorded on the stream the library launches on."""

    def __init__(self):
        self.pairs = []

    def start(self):
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    def stop(self, s):
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        self.pairs.append((s, e))

    def mean_ms(self):
        return sum(s.elapsed_time(e) for s, e in self.pairs) / max(1, len(self.pairs))

    def all_ms(self):
        return [s.elapsed_time(e) for s, e in self.pairs]


def sa_sets(w):
    x = sa_inputs(w["B"], w["T"], w["H"], w["d"], w["seed"], dtype="bf16",
                  lengths=w["lengths"])
    base = {n: x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v", "dout")}
    lengths = x["lengths"].cuda()
    sets = []
    for i in range(N_SETS):
        s = {n: (t if i == 0 else t.clone()) for n, t in base.items()}
        s["out"] = torch.empty_like(s["q"])
        s["lse"] = torch.empty(w["B"], w["H"], w["T"], dtype=torch.float32, device="cuda")
        s["dq"] = torch.empty_like(s["q"])
        s["dk"] = torch.empty_like(s["q"])
        s["dv"] = torch.empty_like(s["q"])
        sets.append(s)
    return sets, lengths, x["lengths"].tolist()


def sa_step(s, lengths, w, tf=None, tb=None, sb=None):
    """Forward on set s, then the backward on set sb (s when None). The timed
    steps give the backward a set whose forward ran two steps earlier, so it
    does not find its q, k, v and out in the Infinity Cache where the forward
    just left them: in a multi-layer training step a layer's backward runs
    long after its forward."""
    sb = s if sb is None else sb
    e = tf.start() if tf else None
    bd.sa_forward(s["q"], s["k"], s["v"], w["Lb"], w["La"], lengths, out=s["out"], lse=s["lse"])
    if tf:
        tf.stop(e)
    e = tb.start() if tb else None
    bd.sa_backward(sb["q"], sb["k"], sb["v"], sb["out"], sb["lse"], sb["dout"], w["Lb"], w["La"],
                   lengths, dq=sb["dq"], dk=sb["dk"], dv=sb["dv"])
    if tb:
        tb.stop(e)


def bench_sa(steps, warmup):
    w = WORKLOAD
    sets, lengths, host_lengths = sa_sets(w)
    # every set's out and lse from its own forward first
    for i in range(N_SETS):
        sa_step(sets[i], lengths, w)
    torch.cuda.synchronize()
    # each step marshalled once: the timed loop issues bare C-ABI calls; step
    # i runs the forward on set i and the backward on set i + 2
    step_calls = [bd.prepared(sa_step, sets[i], lengths, w, sb=sets[(i + 2) % N_SETS])
                  for i in range(N_SETS)]
    ramp(step_calls)
    for i in range(warmup):
        step_calls[i % N_SETS]()
    torch.cuda.synchronize()
    # the timed steps carry no events of their own: an event between two
    # kernels costs more than the gap it measures
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        step_calls[i % N_SETS]()
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    # per-kernel average durations: back-to-back launches of one kernel
    # between two events (the forward rewrites the same out and lse)
    n = min(steps, 50)

    def fwd(s):
        bd.sa_forward(s["q"], s["k"], s["v"], w["Lb"], w["La"], lengths, out=s["out"],
                      lse=s["lse"])

    def bwd(s):
        bd.sa_backward(s["q"], s["k"], s["v"], s["out"], s["lse"], s["dout"], w["Lb"], w["La"],
                       lengths, dq=s["dq"], dk=s["dk"], dv=s["dv"])

    return dict(total_ms=total_ms, fwd_ms=launch_ms(fwd, sets, n),
                bwd_ms=launch_ms(bwd, sets, n), lengths=host_lengths)


def ramp(calls):
    """Issues the calls back to back, in rounds of 50, until RAMP_S seconds of
    wall time have passed with the GPU kept busy."""
    if RAMP_S <= 0:
        return
    t0 = time.perf_counter()
    i = 0
    while True:
        for _ in range(50):
            calls[i % len(calls)]()
            i += 1
        torch.cuda.synchronize()
        if time.perf_counter() - t0 >= RAMP_S:
            return


def launch_ms(fn, sets, n):
    """Average duration of n back-to-back launches, from HIP events recorded on
    the stream the library launches on (the current one). Each set's call is
    marshalled once (binding.prepared), so the loop issues bare C-ABI calls and
    the host keeps ahead of even the shortest kernels."""
    calls = [bd.prepared(fn, s) for s in sets]
    ramp(calls)
    s0 = torch.cuda.Event(enable_timing=True)
    s1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s0.record()
    for i in range(n):
        calls[i % len(calls)]()
    s1.record()
    torch.cuda.synchronize()
    return s0.elapsed_time(s1) / n


def copy_ceiling(mib=64, reps=24):
    """Bandwidth of the library's device-copy reference (sa_copy_reference) at
    the band kernels' traffic size: mib MiB copied (read + written), four
    buffer pairs rotated so no copy finds its source in the Infinity Cache,
    back-to-back launches between HIP events, both access paths."""
    n = mib << 20
    pairs = [(torch.empty(n // 4, dtype=torch.int32, device="cuda"),
              torch.empty(n // 4, dtype=torch.int32, device="cuda")) for _ in range(4)]
    res = {"bytes_copied": n, "bytes_moved": 2 * n}
    for mode, name in ((0, "registers"), (1, "direct_to_lds")):
        for i in range(8):
            bd.copy_reference(*pairs[i % 4], mode)
        ms = launch_ms(lambda p: bd.copy_reference(p[0], p[1], mode), pairs, reps)
        res[name + "_gbs"] = 2 * n / (ms * 1e-3) / 1e9
    res["gbs"] = max(res["registers_gbs"], res["direct_to_lds_gbs"])
    del pairs
    return res


def kernel_floor(reps=200):
    """The per-launch floor of the SA kernels' own launch configuration: the
    workload's B, H, d and window with one frame per sequence and every
    length 0, so each persistent workgroup starts, finds no tile to work on
    and writes one padding row (256 workgroups of 16 (forward) and 12
    (backward) waves, each holding its full LDS allocation), timed back to
    back like the kernels themselves."""
    w = WORKLOAD
    B, H, d = w["B"], w["H"], w["d"]
    z = torch.zeros(B, 1, H, d, dtype=torch.bfloat16, device="cuda")
    t = {n: torch.empty_like(z) for n in ("out", "dq", "dk", "dv")}
    lse = torch.empty(B, H, 1, dtype=torch.float32, device="cuda")
    lengths = torch.zeros(B, dtype=torch.int32, device="cuda")

    def fwd(_):
        bd.sa_forward(z, z, z, w["Lb"], w["La"], lengths, out=t["out"], lse=lse)

    def bwd(_):
        bd.sa_backward(z, z, z, t["out"], lse, z, w["Lb"], w["La"], lengths, dq=t["dq"], dk=t["dk"],
                       dv=t["dv"])
    for f in (fwd, bwd):
        for _ in range(20):
            f(None)
    return {"sa_forward_us": launch_ms(fwd, [None], reps) * 1e3,
            "sa_backward_us": launch_ms(bwd, [None], reps) * 1e3,
            "note": "B=16, T=1, H=12, d=64, Lb=64, La=8, all lengths 0: the launch and "
                    "drain of the persistent grid with no tile to compute"}


C2 = dict(B=8, T=500, H=12, d=64, Lb=32, La=8, lengths="full", seed=2)


def bench_c2(steps, warmup):
    """SA forward bf16 at the paper's l32_r8 window: B=8, T=500 (10 s of 20 ms
    frames), H=12, d=64, Lb=32, La=8, no padding. Twelve copies of the inputs
    rotate (about 300 MB), so no call finds them in the Infinity Cache."""
    c = C2
    x = sa_inputs(c["B"], c["T"], c["H"], c["d"], c["seed"], dtype="bf16", lengths=c["lengths"],
                  with_dout=False)
    base = {n: x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v")}
    lengths = x["lengths"].cuda()
    sets = []
    for i in range(12):
        s = {n: (t if i == 0 else t.clone()) for n, t in base.items()}
        s["out"] = torch.empty_like(s["q"])
        s["lse"] = torch.empty(c["B"], c["H"], c["T"], dtype=torch.float32, device="cuda")
        sets.append(s)

    def fwd(s):
        bd.sa_forward(s["q"], s["k"], s["v"], c["Lb"], c["La"], lengths, out=s["out"],
                      lse=s["lse"])

    for i in range(max(warmup, 12)):
        fwd(sets[i % 12])
    torch.cuda.synchronize()
    ms = launch_ms(fwd, sets, max(steps, 48))
    L = x["lengths"].tolist()
    byts = acc.sa_forward_bytes(L, c["H"], c["d"])
    flops = acc.sa_forward_flops(L, c["H"], c["d"], c["Lb"], c["La"])
    gbs = byts / (ms * 1e-3) / 1e9
    return {
        "workload": "SA forward bf16, B=8, T=500, H=12, d=64, Lb=32, La=8, no padding (the paper's "
                    "l32_r8 window)",
        "ms_per_call": ms,
        "frames_per_s": sum(L) / (ms * 1e-3),
        "useful_tflops": flops / (ms * 1e-3) / 1e12,
        "algorithmic_gbs": gbs,
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
        "algorithmic_bytes": byts,
        "useful_flops": flops,
    }


def bench_llsa(steps, warmup):
    w = WORKLOAD
    x = llsa_inputs(w["B"], w["T"], w["H"], w["d"], 4, dtype="bf16", lengths=w["lengths"],
                    with_dout=True)
    base = {n: x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v", "dout")}
    lengths = x["lengths"].cuda()
    sets = []
    for i in range(N_SETS):
        s = {n: (t if i == 0 else t.clone()) for n, t in base.items()}
        s["out"] = torch.empty_like(s["q"])
        s["lse"] = torch.empty(2, w["B"], w["H"], w["T"], dtype=torch.float32, device="cuda")
        for n in ("dq", "dk", "dv"):
            s[n] = torch.empty_like(s["q"])
        sets.append(s)
    for i in range(warmup):
        s = sets[i % N_SETS]
        bd.llsa_forward(s["q"], s["k"], s["v"], w["Lb"], w["La"], lengths, out=s["out"],
                        lse=s["lse"])
    torch.cuda.synchronize()
    ms = launch_ms(lambda s: bd.llsa_forward(s["q"], s["k"], s["v"], w["Lb"], w["La"], lengths,
                                             out=s["out"], lse=s["lse"]), sets, steps)
    L = x["lengths"].tolist()
    byts = acc.llsa_forward_bytes(L, w["H"], w["d"])
    flops = acc.llsa_forward_flops(L, w["H"], w["d"], w["Lb"], w["La"])

    def bwd(s):
        bd.llsa_backward(s["q"], s["k"], s["v"], s["out"], s["lse"], s["dout"], w["Lb"], w["La"],
                         lengths, dq=s["dq"], dk=s["dk"], dv=s["dv"])

    for i in range(warmup):
        bwd(sets[i % N_SETS])
    torch.cuda.synchronize()
    bms = launch_ms(bwd, sets, steps)
    bbyts = acc.llsa_backward_bytes(L, w["H"], w["d"])
    bflops = acc.llsa_backward_flops(L, w["H"], w["d"], w["Lb"], w["La"])
    backward = {
        "workload": "LLSA backward (two-branch) bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, "
                    "lengths U[400,800]",
        "ms_per_call": bms,
        "frames_per_s": sum(L) / (bms * 1e-3),
        "useful_tflops": bflops / (bms * 1e-3) / 1e12,
        "algorithmic_gbs": bbyts / (bms * 1e-3) / 1e9,
        "roofline": {"bound": "hbm", "achieved": bbyts / (bms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": bbyts / (bms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "traffic": load_traffic("band_bwd_llsa_traffic.json",
                                             source_sha("band_bwd.hip"))},
        "algorithmic_bytes": bbyts,
        "useful_flops": bflops,
    }
    return backward, {
        "workload": "LLSA forward (two-branch) bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, "
                    "lengths U[400,800]",
        "ms_per_call": ms,
        "frames_per_s": sum(L) / (ms * 1e-3),
        "useful_tflops": flops / (ms * 1e-3) / 1e12,
        "algorithmic_gbs": byts / (ms * 1e-3) / 1e9,
        "roofline": {"bound": "hbm", "achieved": byts / (ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": byts / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "traffic": load_traffic("band_fwd_llsa_traffic.json",
                                             source_sha("band_fwd.hip"))},
        "algorithmic_bytes": byts,
        "useful_flops": flops,
    }


def bench_llsa_paper(steps, warmup):
    """The paper's (La+1)-channel LLSA forward and backward on the LLSA
    workload's shapes (nine channels at La = 8)."""
    w = WORKLOAD
    C = w["La"] + 1
    x = llsa_inputs(w["B"], w["T"], w["H"], w["d"], 6, dtype="bf16", lengths=w["lengths"],
                    with_dout=True, channels=C)
    base = {n: x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v", "dout")}
    lengths = x["lengths"].cuda()
    sets = []
    for i in range(N_SETS):
        s = {n: (t if i == 0 else t.clone()) for n, t in base.items()}
        s["out"] = torch.empty_like(s["q"])
        s["lse"] = torch.empty(C, w["B"], w["H"], w["T"], dtype=torch.float32, device="cuda")
        for n in ("dq", "dk", "dv"):
            s[n] = torch.empty_like(s["q"])
        sets.append(s)

    def fwd(s):
        bd.llsa_paper_forward(s["q"], s["k"], s["v"], w["Lb"], w["La"], lengths, out=s["out"],
                              lse=s["lse"])

    def bwd(s):
        bd.llsa_paper_backward(s["q"], s["k"], s["v"], s["out"], s["lse"], s["dout"], w["Lb"],
                               w["La"], lengths, dq=s["dq"], dk=s["dk"], dv=s["dv"])

    for i in range(max(warmup, N_SETS)):
        fwd(sets[i % N_SETS])
    torch.cuda.synchronize()
    ms = launch_ms(fwd, sets, steps)
    for i in range(warmup):
        bwd(sets[i % N_SETS])
    torch.cuda.synchronize()
    bms = launch_ms(bwd, sets, steps)
    L = x["lengths"].tolist()
    rows = {}
    for name, t, byts, flops, traffic in (
            ("forward", ms, acc.llsa_paper_forward_bytes(L, w["H"], w["d"], w["La"]),
             acc.llsa_paper_forward_flops(L, w["H"], w["d"], w["Lb"], w["La"]),
             load_traffic("llsa_paper_fwd_traffic.json", source_sha("band_fwd.hip", "llsa_paper.hip"))),
            ("backward", bms, acc.llsa_paper_backward_bytes(L, w["H"], w["d"], w["La"]),
             acc.llsa_paper_backward_flops(L, w["H"], w["d"], w["Lb"], w["La"]),
             load_traffic("llsa_paper_bwd_traffic.json", source_sha("band_bwd.hip", "llsa_paper.hip")))):
        gbs = byts / (t * 1e-3) / 1e9
        rows[name] = {
            "workload": "LLSA %s, paper form with %d channels, bf16, B=16, T=800, H=12, d=64, "
                        "Lb=64, La=8, lengths U[400,800]" % (name, C),
            "ms_per_call": t,
            "frames_per_s": sum(L) / (t * 1e-3),
            "useful_tflops": flops / (t * 1e-3) / 1e12,
            "algorithmic_gbs": gbs,
            "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": gbs / HBM_PEAK_GBS, "traffic": traffic,
                         "per": "call (all launches of one call)"},
            "algorithmic_bytes": byts,
            "useful_flops": flops,
        }
    return rows["forward"], rows["backward"]


def launch_floor(steps=1000, n_cap=100):
    """What one launch costs by itself: the device-copy reference moving 16
    bytes (one workgroup), launched eagerly with an event pair per launch
    (median) and replayed from a HIP graph of n_cap launches (mean)."""
    src = torch.zeros(4, dtype=torch.int32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(20):
        bd.copy_reference(src, dst)
    torch.cuda.synchronize()
    t = EventTimer()
    for _ in range(steps):
        e = t.start()
        bd.copy_reference(src, dst)
        t.stop(e)
    torch.cuda.synchronize()
    lat = sorted(t.all_ms())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(n_cap):
            bd.copy_reference(src, dst)
    torch.cuda.synchronize()
    g_ms = 0.0
    for _ in range(steps // n_cap):
        s0 = torch.cuda.Event(enable_timing=True)
        s1 = torch.cuda.Event(enable_timing=True)
        s0.record()
        graph.replay()
        s1.record()
        torch.cuda.synchronize()
        g_ms += s0.elapsed_time(s1)
    return {"eager_launch_ms_p50": lat[len(lat) // 2],
            "graph_launch_ms": g_ms / (steps // n_cap * n_cap)}


def stream_roofline(graph_steps_per_s, floor):
    """A streaming step is one launch over a cache-resident working set: its
    bound is the cost of a launch, not HBM. Graph-replayed steps per second
    against the graph-replayed rate of an empty launch."""
    peak = 1.0 / (floor["graph_launch_ms"] * 1e-3)
    return {"bound": "launch", "achieved": graph_steps_per_s, "peak": peak, "unit": "steps/s",
            "frac": graph_steps_per_s / peak, "traffic": None,
            "per": "step (one launch, replayed from a HIP graph)"}


def bench_stream(floor):
    c = STREAM
    S, H, d, Lb, La, steps = c["S"], c["H"], c["d"], c["Lb"], c["La"], c["steps"]
    R = Lb + La + 1
    x = stream_inputs(steps, S, H, d, c["seed"], dtype="bf16")
    q, k, v = (x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v"))
    st = bd.StreamState(S, H, d, Lb, La, R)
    out = torch.empty(S, H, d, dtype=torch.bfloat16, device="cuda")
    # eager, one launch per step, per-step latency from events
    for u in range(20):
        bd.sa_stream_step(st, q[u], k[u], v[u], out=out)
    st = bd.StreamState(S, H, d, Lb, La, R)
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for u in range(steps):
        bd.sa_stream_step(st, q[u], k[u], v[u], out=out)
    end.record()
    torch.cuda.synchronize()
    eager_ms = start.elapsed_time(end)
    # per-step latency, in a pass of its own (an event per step)
    st = bd.StreamState(S, H, d, Lb, La, R)
    t = EventTimer()
    for u in range(steps):
        e = t.start()
        bd.sa_stream_step(st, q[u], k[u], v[u], out=out)
        t.stop(e)
    torch.cuda.synchronize()
    lat = sorted(t.all_ms())
    # graph: capture 100 steps, replay 10 times (the counters advance on the device)
    n_cap = 100
    st = bd.StreamState(S, H, d, Lb, La, R)
    qb = torch.empty(n_cap, S, H, d, dtype=torch.bfloat16, device="cuda")
    kb, vb = torch.empty_like(qb), torch.empty_like(qb)
    side = bd.StreamState(S, H, d, Lb, La, R)
    bd.sa_stream_step(side, q[0], k[0], v[0], out=out)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n_cap):
            bd.sa_stream_step(st, qb[i], kb[i], vb[i], out=out)
    torch.cuda.synchronize()
    g_ms = 0.0
    for r in range(steps // n_cap):
        sl = slice(r * n_cap, (r + 1) * n_cap)
        qb.copy_(q[sl])
        kb.copy_(k[sl])
        vb.copy_(v[sl])
        s0 = torch.cuda.Event(enable_timing=True)
        s1 = torch.cuda.Event(enable_timing=True)
        s0.record()
        graph.replay()
        s1.record()
        torch.cuda.synchronize()
        g_ms += s0.elapsed_time(s1)
    # steady-state step (every stream emitting over a full window)
    widths = [Lb + La + 1] * S
    byts = acc.stream_step_bytes(widths, S, H, d)
    flops = acc.stream_step_flops(widths, H, d)
    mean_step = lat[len(lat) // 2]  # median: a rare host hiccup skews the mean
    return {
        "workload": "SA streaming step bf16, 64 streams x 1000 steps, H=12, d=64, ring 64 past + "
                    "8 look-ahead + current",
        "eager_steps_per_s": steps / (eager_ms * 1e-3),
        "eager_frames_per_s": S * steps / (eager_ms * 1e-3),
        "graph_steps_per_s": steps / (g_ms * 1e-3),
        "graph_frames_per_s": S * steps / (g_ms * 1e-3),
        "step_latency_ms_p50": lat[len(lat) // 2],
        "step_latency_ms_p99": lat[min(len(lat) - 1, int(0.99 * len(lat)))],
        "kernel_gbs_algorithmic": byts / (mean_step * 1e-3) / 1e9,
        "kernel_tflops": flops / (mean_step * 1e-3) / 1e12,
        "roofline": stream_roofline(steps / (g_ms * 1e-3), floor),
        "hbm_frac_algorithmic": byts / (mean_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "launch_floor": floor,
        "note": "ring is L2/MALL resident; the step is launch-bound",
    }


def bench_llsa_stream(floor):
    """llsa_stream_step on the streaming shapes: 64 streams, H=12, d=64, Lb=64,
    La=8, open-ended, every stream emitting both outputs every step after the
    first La steps."""
    c = STREAM
    S, H, d, Lb, La, steps = c["S"], c["H"], c["d"], c["Lb"], c["La"], c["steps"]
    x = stream_inputs(steps, S, H, d, c["seed"], dtype="bf16")
    y = stream_inputs(steps, S, H, d, c["seed"] + 1, dtype="bf16")
    fc = [x[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v")]
    fl = [y[n].to(torch.bfloat16).cuda() for n in ("q", "k", "v")]
    oc = torch.empty(S, H, d, dtype=torch.bfloat16, device="cuda")
    ol = torch.empty_like(oc)

    def step(st, u):
        bd.llsa_stream_step(st, fc[0][u], fc[1][u], fc[2][u], fl[0][u], fl[1][u], fl[2][u],
                            out_c=oc, out_l=ol)

    st = bd.LlsaStreamState(S, H, d, Lb, La)
    for u in range(20):
        step(st, u)
    st = bd.LlsaStreamState(S, H, d, Lb, La)
    torch.cuda.synchronize()
    t = EventTimer()
    for u in range(steps):
        e = t.start()
        step(st, u)
        t.stop(e)
    torch.cuda.synchronize()
    lat = sorted(t.all_ms())
    # graph: capture 100 steps, replay them (the counters advance on the device)
    n_cap = 100
    st = bd.LlsaStreamState(S, H, d, Lb, La)
    bufs = [torch.empty(n_cap, S, H, d, dtype=torch.bfloat16, device="cuda") for _ in range(6)]
    side = bd.LlsaStreamState(S, H, d, Lb, La)
    step(side, 0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(n_cap):
            bd.llsa_stream_step(st, *[b[i] for b in bufs], out_c=oc, out_l=ol)
    torch.cuda.synchronize()
    g_ms = 0.0
    for r in range(steps // n_cap):
        sl = slice(r * n_cap, (r + 1) * n_cap)
        for b, src in zip(bufs, fc + fl):
            b.copy_(src[sl])
        s0 = torch.cuda.Event(enable_timing=True)
        s1 = torch.cuda.Event(enable_timing=True)
        s0.record()
        graph.replay()
        s1.record()
        torch.cuda.synchronize()
        g_ms += s0.elapsed_time(s1)
    widths = [Lb + La + 1] * S
    byts = acc.llsa_stream_step_bytes(widths, S, H, d)
    flops = acc.llsa_stream_step_flops(widths, H, d)
    mean_step = lat[len(lat) // 2]  # median: a rare host hiccup skews the mean
    return {
        "workload": "LLSA (two-branch) streaming step bf16, 64 streams x 1000 steps, H=12, d=64, "
                    "rings of 64 past + 8 look-ahead + current frames per branch",
        "graph_steps_per_s": (steps // n_cap * n_cap) / (g_ms * 1e-3),
        "graph_frames_per_s": S * (steps // n_cap * n_cap) / (g_ms * 1e-3),
        "step_latency_ms_p50": lat[len(lat) // 2],
        "step_latency_ms_p99": lat[min(len(lat) - 1, int(0.99 * len(lat)))],
        "kernel_gbs_algorithmic": byts / (mean_step * 1e-3) / 1e9,
        "kernel_tflops": flops / (mean_step * 1e-3) / 1e12,
        "roofline": stream_roofline((steps // n_cap * n_cap) / (g_ms * 1e-3), floor),
        "hbm_frac_algorithmic": byts / (mean_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "launch_floor": floor,
        "note": "two outputs per stream and step; the rings are L2/MALL resident; launch-bound",
    }


STACK = dict(layers=12, S=64, H=12, d=64, Lb=64, La=(8, 16), T=200, frame_ms=20.0, seed=9)


def bench_stream_latency():
    """Algorithmic latency of a 12-layer streaming stack (Tab. 3): the step at
    which the top layer emits each frame, SA against LLSA, and the wall time
    of one step of the whole stack."""
    from paper_2302_13451_amd.streaming import StackedStream

    c = STACK
    L, S, H, d, Lb, T = c["layers"], c["S"], c["H"], c["d"], c["Lb"], c["T"]
    g = torch.Generator(device="cpu").manual_seed(c["seed"])
    W = [torch.randn(3, H * d, H * d, generator=g) / math.sqrt(H * d) for _ in range(L)]
    x = torch.randn(T, S, H, d, generator=g).to(torch.bfloat16).cuda()
    res = {"workload": "%d-layer streaming stack, %d streams of %d frames, H=%d, d=%d, Lb=%d, "
                       "La=%s, bf16, random projections; %g ms per frame"
                       % (L, S, T, H, d, Lb, "/".join(str(a) for a in c["La"]), c["frame_ms"])}
    for La in c["La"]:
        for kind in ("sa", "llsa"):
            model = StackedStream(kind, W, S, H, d, Lb, La, lengths=[T] * S)
            t = EventTimer()
            lag = []
            for n in range(T + L * La):
                e = t.start()
                _, em = model.step(x[n] if n < T else None)
                t.stop(e)
                f = int(em[0])
                if f >= 0:
                    lag.append(n - f)
            torch.cuda.synchronize()
            ms = sorted(t.all_ms())
            frames = max(lag)
            res["%s_La%d" % (kind, La)] = {
                "algorithmic_latency_frames": frames,
                "algorithmic_latency_s": frames * c["frame_ms"] * 1e-3,
                "latency_constant_over_frames": min(lag) == frames and len(lag) == T,
                "stack_step_ms_p50": ms[len(ms) // 2],
                "stack_step_ms_p99": ms[min(len(ms) - 1, int(0.99 * len(ms)))],
            }
    return res


def bench_masked_attention(steps=5):
    """Masked full attention (dense T x T scores + band mask) in PyTorch,
    forward+backward, bf16 inputs with float32 softmax, same workload."""
    w = WORKLOAD
    x = sa_inputs(w["B"], w["T"], w["H"], w["d"], w["seed"], dtype="bf16", lengths=w["lengths"])
    T = w["T"]
    t = torch.arange(T, device="cuda")
    L = x["lengths"].cuda()
    band = (t[None, :] >= t[:, None] - w["Lb"]) & (t[None, :] <= t[:, None] + w["La"])
    mask = band[None, None] & (t[None, None, None, :] < L[:, None, None, None])
    rows = (t[None, :] < L[:, None])[:, None, :, None]
    q, k, v, do = (x[n].to(torch.bfloat16).cuda().permute(0, 2, 1, 3).contiguous()
                   for n in ("q", "k", "v", "dout"))

    def step():
        qq, kk, vv = (a.detach().requires_grad_(True) for a in (q, k, v))
        s = torch.matmul(qq.float(), kk.float().transpose(-1, -2).contiguous()) / math.sqrt(w["d"])
        s = s.masked_fill(~mask, float("-inf"))
        p = torch.softmax(s, dim=-1)
        p = torch.where(rows, p, torch.zeros_like(p))
        o = torch.matmul(p, vv.float())
        o.backward(do.float())
        return o

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    s0 = torch.cuda.Event(enable_timing=True)
    s1 = torch.cuda.Event(enable_timing=True)
    s0.record()
    for _ in range(steps):
        step()
    s1.record()
    torch.cuda.synchronize()
    ms = s0.elapsed_time(s1) / steps
    frames = sum(x["lengths"].tolist())
    res = {"workload": "masked full attention fwd+bwd in PyTorch (float32 math on bf16 inputs), "
                       "same batch", "ms_per_step": ms, "frames_per_s": frames / (ms * 1e-3)}
    # torch's scaled_dot_product_attention with the boolean band mask (padded
    # query rows keep their own frame so no row is empty; their output is
    # zeroed). float32 operands: its bfloat16 paths are not used here.
    sdpa_mask = mask | (t[None, :] == t[:, None])[None, None]

    def sdpa_step():
        qq, kk, vv = (a.float().detach().requires_grad_(True) for a in (q, k, v))
        o = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, attn_mask=sdpa_mask)
        o = torch.where(rows, o, torch.zeros_like(o))
        o.backward(do.float())
        return o

    try:
        for _ in range(2):
            sdpa_step()
        torch.cuda.synchronize()
        s0.record()
        for _ in range(steps):
            sdpa_step()
        s1.record()
        torch.cuda.synchronize()
        sms = s0.elapsed_time(s1) / steps
        res["sdpa_bool_mask"] = {"workload": "torch scaled_dot_product_attention fwd+bwd with a "
                                             "boolean band attn_mask, float32, same batch",
                                 "ms_per_step": sms, "frames_per_s": frames / (sms * 1e-3)}
    except RuntimeError as e:
        res["sdpa_bool_mask"] = {"error": str(e)[:200]}
    return res


MEMORY_EXPERIMENT = {"B": 4, "T": 1000, "d": 64, "heads": (8, 16), "La": 8,
                     "widths": tuple(range(10, 491, 40))}


def _peak_bytes(fn):
    """Peak bytes the caching allocator hands out while fn runs, above what
    was allocated when it started (fn allocates its own inputs)."""
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.reset_peak_memory_stats()
    base = torch.cuda.memory_allocated()
    fn()
    torch.cuda.synchronize()
    return torch.cuda.max_memory_allocated() - base


def sa_training_memory(B, T, H, d, Lb, La):
    """Peak memory of one SA layer's forward + backward through the library:
    q, k, v and dout, out and lse, dq, dk and dv (bf16, lse float32). The
    kernels allocate nothing, so this is the tensors themselves."""
    def run():
        g = torch.Generator(device="cuda").manual_seed(7)
        q, k, v, do = (torch.empty(B, T, H, d, dtype=torch.bfloat16, device="cuda").normal_(generator=g)
                       for _ in range(4))
        out, lse = bd.sa_forward(q, k, v, Lb, La)
        dq, dk, dv = bd.sa_backward(q, k, v, out, lse, do, Lb, La)
        torch.cuda.synchronize()
        del q, k, v, do, out, lse, dq, dk, dv
    return _peak_bytes(run)


def sa_tensors_memory(B, T, H, d):
    """Peak memory of allocating the same tensors as sa_training_memory, in the
    same order, with no kernel run: what the allocator's rounding makes of
    them."""
    def run():
        ts = [torch.empty(B, T, H, d, dtype=torch.bfloat16, device="cuda") for _ in range(5)]
        ts.append(torch.empty(B, H, T, dtype=torch.float32, device="cuda"))
        ts += [torch.empty(B, T, H, d, dtype=torch.bfloat16, device="cuda") for _ in range(3)]
        torch.cuda.synchronize()
        del ts
    return _peak_bytes(run)


def maa_training_memory(B, T, H, d, Lb, La):
    """Peak memory of masked acausal attention (the paper's MAA: dense T x T
    scores, band mask) forward + backward with PyTorch autograd, on the same
    bf16 tensors, float32 scores and softmax."""
    def run():
        g = torch.Generator(device="cuda").manual_seed(7)
        q, k, v, do = (torch.empty(B, H, T, d, dtype=torch.bfloat16, device="cuda").normal_(generator=g)
                       for _ in range(4))
        t = torch.arange(T, device="cuda")
        mask = (t[None, :] >= t[:, None] - Lb) & (t[None, :] <= t[:, None] + La)
        qq, kk, vv = (a.detach().requires_grad_(True) for a in (q, k, v))
        s_ = torch.matmul(qq.float(), kk.float().transpose(-1, -2).contiguous()) / math.sqrt(d)
        s_ = s_.masked_fill(~mask, float("-inf"))
        p = torch.softmax(s_, dim=-1)
        o = torch.matmul(p, vv.float()).to(torch.bfloat16)
        o.backward(do)
        torch.cuda.synchronize()
        del q, k, v, do, qq, kk, vv, s_, p, o, mask
    return _peak_bytes(run)


def memory_experiment():
    """Memory per training vector (one sequence) of one attention layer's
    forward + backward against the receptive field W = Lb + La + 1, SA through
    the library against MAA in PyTorch (Sec. "Lower Memory Usage", Fig. 5),
    at d = 64, N_T = 1000, H = 8 and 16, La = 8."""
    c = MEMORY_EXPERIMENT
    B, T, d, La = c["B"], c["T"], c["d"], c["La"]
    maa_training_memory(B, T, c["heads"][0], d, 9, La)  # first-call workspaces of the library GEMMs
    rows = []
    for H in c["heads"]:
        for W in c["widths"]:
            Lb = W - 1 - La
            sa = sa_training_memory(B, T, H, d, Lb, La)
            maa = maa_training_memory(B, T, H, d, Lb, La)
            rows.append({"H": H, "W": W, "Lb": Lb, "La": La, "sa_bytes_per_vector": sa / B,
                         "maa_bytes_per_vector": maa / B,
                         "sa_tensors_allocated_per_vector": sa_tensors_memory(B, T, H, d) / B,
                         "sa_tensor_bytes_per_vector": acc.sa_training_tensor_bytes(T, H, d)})
    return {"experiment": "memory per training vector, one attention layer forward+backward, "
                          "B=%d, T=%d, d=%d, bf16 tensors" % (B, T, d), "rows": rows}


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _timed_passes(fn, min_seconds):
    passes, t0 = 0, time.perf_counter()
    while True:
        fn()
        passes += 1
        el = time.perf_counter() - t0
        if el >= min_seconds:
            return passes, el


def cpu_baseline(min_seconds=10.0):
    """The fp64 oracle (plain C, OpenMP over (sequence, head)) on the host:
    repeated forward+backward passes over the workload's sequences with every
    core the process may run on, then on one core, then the other configs'
    passes (short samples)."""
    import oracle

    oracle._load()
    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    w = WORKLOAD
    x = sa_inputs(w["B"], w["T"], w["H"], w["d"], w["seed"], dtype="bf16", lengths=w["lengths"])
    q, k, v, do = (x[n].double().numpy() for n in ("q", "k", "v", "dout"))
    ln = x["lengths"].numpy()

    def step(nseq, threads):
        oracle.sa_forward(q[:nseq], k[:nseq], v[:nseq], w["Lb"], w["La"], ln[:nseq],
                          threads=threads)
        oracle.sa_backward(q[:nseq], k[:nseq], v[:nseq], do[:nseq], w["Lb"], w["La"], ln[:nseq],
                           threads=threads)

    passes, el = _timed_passes(lambda: step(w["B"], cores), min_seconds)
    frames = int(ln.sum()) * passes
    res = {"value": frames / el, "unit": "frames/s", "cores": cores, "kind": "oracle",
           "sample": "%d passes of forward+backward over the whole workload batch (16 sequences, "
                     "%d frames, 12 heads), %.1f s" % (passes, int(ln.sum()), el),
           "cpu_model": _cpu_model(), "host_cpus": os.cpu_count()}
    p1, el1 = _timed_passes(lambda: step(1, 1), min_seconds / 4)
    res["one_core"] = {"value": int(ln[0]) * p1 / el1, "unit": "frames/s", "cores": 1,
                       "sample": "%d passes over the first sequence (%d frames), %.1f s"
                                 % (p1, int(ln[0]), el1)}
    # the other configurations, all cores, short samples
    c = C2
    y = sa_inputs(c["B"], c["T"], c["H"], c["d"], c["seed"], dtype="bf16", lengths=c["lengths"],
                  with_dout=False)
    yq, yk, yv = (y[n].double().numpy() for n in ("q", "k", "v"))
    pc, elc = _timed_passes(lambda: oracle.sa_forward(yq, yk, yv, c["Lb"], c["La"], None,
                                                      threads=cores), min_seconds / 4)
    res["sa_forward_l32_r8"] = {"value": c["B"] * c["T"] * pc / elc, "unit": "frames/s",
                                "cores": cores, "sample": "%d forward passes, B=8, T=500, %.1f s"
                                                          % (pc, elc)}
    z = llsa_inputs(w["B"], w["T"], w["H"], w["d"], 4, dtype="bf16", lengths=w["lengths"])
    zq, zk, zv = (z[n].double().numpy() for n in ("q", "k", "v"))
    zl = z["lengths"].numpy()
    pl, ell = _timed_passes(lambda: oracle.llsa_two_branch(zq, zk, zv, w["Lb"], w["La"], zl,
                                                           threads=cores), min_seconds / 4)
    res["llsa_forward"] = {"value": int(zl.sum()) * pl / ell, "unit": "frames/s", "cores": cores,
                           "sample": "%d passes of the two-branch forward over the LLSA batch, "
                                     "%.1f s" % (pl, ell)}
    st = STREAM
    S, H, d, Lb, La = st["S"], st["H"], st["d"], st["Lb"], st["La"]
    sx = stream_inputs(200, S, H, d, st["seed"], dtype="bf16")
    so = oracle.StreamOracle(S, H, d, Lb, La, Lb + La + 1)
    sq, sk, sv = (sx[n].double().numpy() for n in ("q", "k", "v"))
    n_st, t0 = 0, time.perf_counter()
    while time.perf_counter() - t0 < min_seconds / 4 and n_st < 200:
        so.step(sq[n_st], sk[n_st], sv[n_st])
        n_st += 1
    els = time.perf_counter() - t0
    res["stream_step"] = {"value": n_st / els, "unit": "steps/s", "cores": 1,
                          "sample": "%d streaming steps of 64 streams (the oracle's ring "
                                    "simulation runs on one core), %.1f s" % (n_st, els)}
    return res


def main():
    global RAMP_S
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="time only the SA forward+backward step")
    ap.add_argument("--no-stack", action="store_true",
                    help="skip the streaming-stack latency row (its many small launches crowd "
                         "kernel traces)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of 512 MiB (counter calibration)")
    ap.add_argument("--memory-experiment", action="store_true",
                    help="only measure memory per training vector, SA against masked attention")
    ap.add_argument("--ramp-ms", type=float, default=RAMP_S * 1e3,
                    help="milliseconds of back-to-back launches before every timed loop (0 for "
                         "profiler runs, whose per-dispatch records it would multiply)")
    args = ap.parse_args()
    RAMP_S = max(0.0, args.ramp_ms) * 1e-3
    if args.gpus != 1:
        print("bench.py runs on one GPU only: --gpus %d is not supported (the band kernels shard "
              "over batch and heads with no communication)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        # the library's device-copy reference, 512 MiB, five launches through
        # registers, then five through direct global->LDS copies
        bd.load_library()
        n = 512 << 20
        src = torch.ones(n // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        for mode in (0, 1):
            for _ in range(5):
                bd.copy_reference(src, dst, mode)
            torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches_per_mode": 5}))
        return
    bd.load_library()
    if args.memory_experiment:
        print(json.dumps(memory_experiment()), flush=True)
        return
    log("SA forward+backward: %d warmup + %d timed steps" % (args.warmup, args.steps))
    r = bench_sa(args.steps, args.warmup)
    w = WORKLOAD
    L = r["lengths"]
    frames = sum(L)
    step_s = r["total_ms"] * 1e-3 / args.steps
    fwd_b = acc.sa_forward_bytes(L, w["H"], w["d"])
    bwd_b = acc.sa_backward_bytes(L, w["H"], w["d"])
    fwd_f = acc.sa_forward_flops(L, w["H"], w["d"], w["Lb"], w["La"])
    bwd_f = acc.sa_backward_flops(L, w["H"], w["d"], w["Lb"], w["La"])
    fwd_gbs = fwd_b / (r["fwd_ms"] * 1e-3) / 1e9
    bwd_gbs = bwd_b / (r["bwd_ms"] * 1e-3) / 1e9
    dominant = "sa_backward" if r["bwd_ms"] >= r["fwd_ms"] else "sa_forward"
    dom_gbs = bwd_gbs if dominant == "sa_backward" else fwd_gbs
    dom_sha = source_sha("band_bwd.hip") if dominant == "sa_backward" else source_sha("band_fwd.hip")
    traffic_file = ("sa_bwd_traffic.json" if dominant == "sa_backward" else "sa_fwd_traffic.json")
    sq_file = ("sa_bwd_sq_counters.json" if dominant == "sa_backward" else "sa_fwd_sq_counters.json")
    line = {
        "metric": "band-attention frames/s + TFLOP/s & HBM GB/s vs roofline (fwd+bwd)",
        "value": frames / step_s,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "clock_ramp_ms": RAMP_S * 1e3,
        "ms_per_step": r["total_ms"] / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "SA forward+backward bf16, B=16, T=800, H=12, d=64, Lb=64, La=8, "
                               "lengths U[400,800] (20 ms frames)",
                   "B": w["B"], "T": w["T"], "H": w["H"], "d": w["d"], "Lb": w["Lb"],
                   "La": w["La"], "valid_frames": frames, "input_sets_rotated": N_SETS},
        "roofline": {"bound": "hbm", "achieved": dom_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": dom_gbs / HBM_PEAK_GBS, "kernel": dominant,
                     "traffic": load_traffic(traffic_file, dom_sha),
                     "mfma": load_mfma(sq_file, dom_sha)},
        "kernels": {
            "sa_forward": {"ms": r["fwd_ms"], "algorithmic_bytes": fwd_b, "gbs": fwd_gbs,
                           "hbm_frac": fwd_gbs / HBM_PEAK_GBS, "useful_flops": fwd_f,
                           "tflops": fwd_f / (r["fwd_ms"] * 1e-3) / 1e12},
            "sa_backward": {"ms": r["bwd_ms"], "algorithmic_bytes": bwd_b, "gbs": bwd_gbs,
                            "hbm_frac": bwd_gbs / HBM_PEAK_GBS, "useful_flops": bwd_f,
                            "tflops": bwd_f / (r["bwd_ms"] * 1e-3) / 1e12},
        },
        "useful_tflops_step": (fwd_f + bwd_f) / step_s / 1e12,
        "algorithmic_gbs_step": (fwd_b + bwd_b) / step_s / 1e9,
    }
    log("device-copy reference (practical bandwidth ceiling)")
    ceiling = copy_ceiling()
    line["copy_ceiling"] = ceiling
    line["roofline"]["copy_ceiling_gbs"] = ceiling["gbs"]
    line["roofline"]["practical_frac"] = dom_gbs / ceiling["gbs"]
    log("launch floor of the SA kernels' configuration")
    floor_k = kernel_floor()
    line["kernel_launch_floor"] = floor_k
    line["roofline"]["launch_floor_us"] = floor_k["sa_backward_us" if dominant == "sa_backward"
                                                  else "sa_forward_us"]
    if not args.no_extras:
        log("SA forward at the l32_r8 window (B=8, T=500)")
        line["sa_forward_l32_r8"] = bench_c2(args.steps, args.warmup)
        log("LLSA forward and backward")
        line["llsa_backward"], line["llsa"] = bench_llsa(max(20, args.steps // 2), 5)
        log("LLSA in the paper's channel form, forward and backward")
        line["llsa_paper"], line["llsa_paper_backward"] = bench_llsa_paper(20, 3)
        log("launch floor")
        floor = launch_floor()
        log("streaming step")
        line["stream"] = bench_stream(floor)
        log("LLSA streaming step")
        line["llsa_stream"] = bench_llsa_stream(floor)
        if not args.no_stack:
            log("12-layer streaming stack latency")
            line["stream_latency"] = bench_stream_latency()
        log("masked full attention in PyTorch")
        try:
            line["masked_attention_torch"] = bench_masked_attention()
        except RuntimeError as e:  # e.g. out of memory on a smaller card
            line["masked_attention_torch"] = {"error": str(e)[:200]}
    if not args.no_cpu_baseline:
        log("CPU oracle baseline")
        line["cpu_baseline"] = cpu_baseline()
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
