#!/usr/bin/env python3
"""Benchmark of the Gorila DQN learner step on one MI355X.

A step is one whole learner step (Algorithm 1 of Nair et al. 2015): gather the
minibatch out of replay, online and target Q forward passes, TD target and
Huber-clipped TD error, loss, and backprop to every parameter gradient.  The
timed workload is the batch-512, 6-action fp32 step on seeded synthetic
Atari-shaped data (uint8 4x84x84 stacks); inputs sit in HBM before timing.

Prints one JSON line: transitions/s, the fraction of fp32 MFMA peak the whole
step reaches, the roofline of the dominant kernel (timed live with HIP events
on the stream the kernels run on) and the fp64 CPU oracle timed on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP32_MFMA_PEAK_TFLOPS = 157.3   # MI355X dense fp32 matrix peak
BF16_MFMA_PEAK_TFLOPS = 2516.6  # MI355X dense bf16 matrix peak
HBM_PEAK_GBS = 8000.0

# Algorithmic multiply-accumulates per sample of each layer (Section 5.1 net).
MAC_CONV1 = 400 * 32 * 256
MAC_CONV2 = 81 * 64 * 512
MAC_CONV3 = 49 * 64 * 576
MAC_FC1 = 3136 * 512


def step_flops_per_transition(A: int) -> int:
    """Online + target forward, data gradients of layers 2-5, weight gradients
    of layers 1-5; the action head's backward counted at the chosen action."""
    fwd = MAC_CONV1 + MAC_CONV2 + MAC_CONV3 + MAC_FC1 + 512 * A
    bwd = 2 * 512 + 2 * MAC_FC1 + 2 * MAC_CONV3 + 2 * MAC_CONV2 + MAC_CONV1
    return 2 * (2 * fwd + bwd)


MFMA_STAGES = ("conv1_fwd", "conv2_fwd", "conv3_fwd", "fc1_fwd", "fc1_bwd", "conv3_bwd",
               "conv2_bwd", "conv1_wgrad")


def stage_flops(stage: str, B: int, A: int) -> float:
    """Algorithmic FLOPs of one launch of a stage of the learner step at batch B
    (the backward stages each hold a data gradient and a weight gradient)."""
    two = 2 * B  # online + target rows in the forward stages
    table = {
        "conv1_fwd": two * MAC_CONV1, "conv2_fwd": two * MAC_CONV2, "conv3_fwd": two * MAC_CONV3,
        "fc1_fwd": two * MAC_FC1, "head": two * 512 * A + B * 512,
        "fc1_bwd": 2 * B * MAC_FC1 + B * 512, "conv3_bwd": 2 * B * MAC_CONV3,
        "conv2_bwd": 2 * B * MAC_CONV2, "conv1_wgrad": B * MAC_CONV1,
    }
    return 2.0 * table.get(stage, 0)


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "traffic_learner_b512_a6.json")
STATS_PROFILE = os.path.join(ROOT, "profiles", "learner_b512_a6_kernel_stats.json")


def library_digest() -> str:
    """sha256 of the built libgorila.so: the kernels the counters were taken on."""
    import hashlib
    import paper_1507_04296_amd as g
    return hashlib.sha256(open(g.LIB_PATH, "rb").read()).hexdigest()


def stored_traffic(stage: str, B: int, A: int):
    """HBM bytes per launch of `stage` from the committed rocprofv3 FETCH_SIZE /
    WRITE_SIZE runs, scaled by the copy calibration; None when the library has
    been rebuilt differently since those counters were taken, or for another
    workload."""
    try:
        prof = json.load(open(TRAFFIC_PROFILE))
    except (OSError, ValueError):
        return None
    if prof.get("library_sha256") != library_digest() or prof.get("batch") != B \
            or prof.get("n_actions") != A or stage not in prof.get("kernels", {}):
        return None
    k = prof["kernels"][stage]
    return (k["fetch_kib"] / prof["copy_fetch_factor"] +
            k["write_kib"] / prof["copy_write_factor"]) * 1024.0


def stored_launch_ms(stage: str, B: int, A: int):
    """(average ms per launch of `stage`, profile file) from the committed
    rocprofv3 kernel statistics, or None when the library has been rebuilt
    differently since they were taken, or for another workload."""
    try:
        prof = json.load(open(STATS_PROFILE))
    except (OSError, ValueError):
        return None
    if prof.get("library_sha256") != library_digest() or prof.get("batch") != B \
            or prof.get("n_actions") != A or stage not in prof.get("stages", {}):
        return None
    return prof["stages"][stage]["avg_us"] / 1e3, os.path.relpath(STATS_PROFILE, ROOT)


def host_cpu():
    """The host's CPU model and core counts (for the CPU baseline)."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cpus": usable}


def step_percentiles(torch, fn, steps):
    """p10 / p50 / p90 of per-call times (ms): one event between consecutive
    calls on the current stream (a separate pass from the headline timing)."""
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    evs[0].record()
    for i in range(steps):
        fn()
        evs[i + 1].record()
    torch.cuda.synchronize()
    per = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(steps)])
    return [round(float(x), 4) for x in np.percentile(per, [10, 50, 90])]


def time_region(torch, fn, steps):
    """Mean ms per call over `steps` calls bracketed by two events."""
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


SETTLE_S = 0.3


def settle(torch, fn, seconds=SETTLE_S):
    """Untimed calls until `seconds` of wall time have passed (after the W
    warm-up calls): the GPU's clocks ramp up over milliseconds of load, and a
    handful of sub-millisecond warm-up steps leaves the timed steps on a GPU
    that is still speeding up.  The figure sought is the steady-state rate of
    a learner that runs continuously."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(16):
            fn()
        torch.cuda.synchronize()


def run_learner(torch, g, datagen, B, A, seed, steps, warmup, timed_stage=None, graph=False):
    inp = datagen.learner_inputs(seed, B, A)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    theta, tgt, idx = t(inp.theta), t(inp.theta_target), t(inp.idx)
    rep = g.Replay.stacked(t(inp.s), t(inp.s2), t(inp.a), t(inp.r), t(inp.term))
    ctx = g.Context(B, A, device=dev)
    grads = torch.empty(g.param_count(A), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    step = lambda: g.gorila_learner_step(ctx, theta, tgt, A, rep, idx, inp.gamma, 1.0, grads, loss)
    for _ in range(warmup):
        step()
    settle(torch, step)
    ctx.check()

    # per-stage profile (separate pass, every stage bracketed by events)
    names = g.stage_names()
    ctx.timing_begin(names, max_records=len(names) * max(steps, 1))
    for _ in range(max(steps // 2, 1)):
        step()
    prof = ctx.timing_end()

    dominant = timed_stage or max((k for k in prof if k in MFMA_STAGES), key=lambda k: prof[k][0])
    # timed region: events only around the dominant kernel, on the first
    # quarter of the timed steps (each event pair costs the step a few
    # microseconds; the kernel's average over those launches is the figure)
    torch.cuda.synchronize()
    ctx.timing_begin([dominant], max_records=max(1, steps // 4))
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom = ctx.timing_end()[dominant]
    ctx.check()
    ms_total = start.elapsed_time(stop)
    pct = step_percentiles(torch, step, steps)
    graph_ms = None
    if graph:
        # the same step captured once into a HIP graph and replayed
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            step()
        for _ in range(warmup):
            gr.replay()
        graph_ms = time_region(torch, gr.replay, steps)
        ctx.bind_stream()
        ctx.check()
    ctx.close()
    return dict(inp=inp, ms_per_step=ms_total / steps, wall_s=wall, prof=prof, dominant=dominant,
                dominant_ms=dom[0] / max(dom[1], 1), dominant_launches=dom[1], pct=pct,
                graph_ms=graph_ms)


def run_two_learners(torch, g, datagen, B, A, seed, steps, warmup):
    """Two independent learners (their own contexts and gradient buffers, the
    same minibatch) stepping on two streams at once, as learners bundled on one
    GPU would: the learner transitions/s of the pair, timed from one event on
    the current stream to the join of both streams."""
    inp = datagen.learner_inputs(seed, B, A)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    theta, tgt, idx = t(inp.theta), t(inp.theta_target), t(inp.idx)
    rep = g.Replay.stacked(t(inp.s), t(inp.s2), t(inp.a), t(inp.r), t(inp.term))
    streams = [torch.cuda.Stream(device=dev) for _ in range(2)]  # default priority
    learners = []
    for s in streams:
        with torch.cuda.stream(s):
            learners.append((g.Context(B, A, device=dev),
                             torch.empty(g.param_count(A), dtype=torch.float32, device=dev),
                             torch.empty(1, dtype=torch.float32, device=dev)))
    def step_pair():
        for s, (ctx, grads, loss) in zip(streams, learners):
            with torch.cuda.stream(s):
                g.gorila_learner_step(ctx, theta, tgt, A, rep, idx, inp.gamma, 1.0, grads, loss)
    for _ in range(warmup):
        step_pair()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cur = torch.cuda.current_stream(dev)
    start.record(cur)
    for s in streams:
        s.wait_event(start)
    for _ in range(steps):
        step_pair()
    for s in streams:
        cur.wait_stream(s)
    stop.record(cur)
    torch.cuda.synchronize()
    for ctx, _, _ in learners:
        ctx.check()
        ctx.close()
    ms_per_step = start.elapsed_time(stop) / (2 * steps)
    return {"workload": f"learner_b{B}_a{A}_f32 x 2 learners", "streams": 2,
            "value": round(B / (ms_per_step * 1e-3), 1), "unit": "transitions/s",
            "ms_per_learner_step": round(ms_per_step, 4),
            "note": "two independent learner steps in flight at once (bundled learners); "
                    "not the headline value, which times one learner's steps back to back"}


def run_grouped(torch, g, datagen, steps, warmup):
    """The stale-replica workload: 16 bf16 replicas x 64 transitions, 18 actions."""
    w = datagen.WORKLOADS["grouped_g16_b64_a18_bf16"]
    G, b, A = w["groups"], w["batch"], w["n_actions"]
    inp = datagen.grouped_inputs(w["seed"], G, b, A)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    thetas, tgt = t(inp.theta_bf16.view(np.int16)), t(inp.target_bf16.view(np.int16))
    idx = torch.arange(G * b, dtype=torch.int64, device=dev)
    rep = g.Replay.stacked(t(inp.s), t(inp.s2), t(inp.a), t(inp.r), t(inp.term))
    ctx = g.Context(b, A, groups=G, device=dev, dtype=g.GORILA_BF16)
    grads = torch.empty((G, g.param_count(A)), dtype=torch.float32, device=dev)
    loss = torch.empty(G, dtype=torch.float32, device=dev)
    step = lambda: g.gorila_learner_step_grouped(ctx, thetas, tgt, A, rep, idx, b, inp.gamma, 1.0,
                                                 grads, loss)
    for _ in range(warmup):
        step()
    ctx.check()
    names = g.stage_names()
    ctx.timing_begin(names, max_records=len(names) * G * max(steps, 1))
    for _ in range(max(steps // 2, 1)):
        step()
    prof = ctx.timing_end()
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        step()
    stop.record()
    torch.cuda.synchronize()
    ctx.check()
    ms = start.elapsed_time(stop) / steps
    ctx.close()
    n = max(steps // 2, 1)
    tflops = G * b * step_flops_per_transition(A) / (ms * 1e-3) / 1e12
    # every parameter set is bf16, so the products run on bf16 MFMA operands
    # (forward activations as two bf16 terms) with fp32 accumulation; tflops
    # counts algorithmic FLOPs, priced against the dense bf16 peak
    # compulsory HBM bytes of the step: both stacks of every transition, the G
    # bf16 replicas and the bf16 target read once, the G fp32 gradients written
    P = g.param_count(A)
    compulsory = 2 * G * b * datagen.STATE_BYTES + (G + 1) * P * 2 + G * P * 4
    hbm_tbs = compulsory / (ms * 1e-3) / 1e12
    mfma_s = G * b * step_flops_per_transition(A) / (BF16_MFMA_PEAK_TFLOPS * 1e12)
    hbm_s = compulsory / (HBM_PEAK_GBS * 1e9)
    return {"workload": "grouped_g16_b64_a18_bf16", "value": round(G * b / (ms * 1e-3), 1),
            "unit": "transitions/s", "ms_per_step": round(ms, 4), "tflops": round(tflops, 2),
            "dtype": "bf16 operands, f32 accumulation",
            "pct_mfma_peak": round(100 * tflops / BF16_MFMA_PEAK_TFLOPS, 2),
            "mfma_peak_tflops": BF16_MFMA_PEAK_TFLOPS,
            "roofline": {"mfma_bf16": {"floor_ms": round(mfma_s * 1e3, 4),
                                       "frac": round(tflops / BF16_MFMA_PEAK_TFLOPS, 4)},
                         "hbm": {"compulsory_bytes": compulsory, "floor_ms": round(hbm_s * 1e3, 4),
                                 "achieved_tb_per_s": round(hbm_tbs, 3),
                                 "frac": round(hbm_tbs * 1e3 / HBM_PEAK_GBS, 4)},
                         "binding": "hbm" if hbm_s > mfma_s else "mfma"},
            "stage_ms": {k: round(v[0] / n, 4) for k, v in prof.items()}}


def run_actor(torch, g, datagen, steps, warmup):
    """Actor inference: Q forward + epsilon-greedy for 1024 environments, 18 actions."""
    w = datagen.WORKLOADS["actor_n1024_a18_f32"]
    n, A = w["n"], w["n_actions"]
    inp = datagen.actor_inputs(w["seed"], n, A, w["eps"])
    dev = torch.device("cuda:0")
    theta = torch.from_numpy(inp.theta).to(dev)
    states = torch.from_numpy(np.ascontiguousarray(inp.states)).to(dev)
    ctx = g.Context((n + 1) // 2, A, device=dev)
    acts = torch.empty(n, dtype=torch.int32, device=dev)
    q = torch.empty((n, A), dtype=torch.float32, device=dev)
    call = lambda: g.gorila_act(ctx, theta, A, states, inp.eps, inp.seed, acts, q)
    for _ in range(warmup):
        call()
    ctx.check()
    ms = time_region(torch, call, steps)
    ctx.check()
    # storing the step: one record into each of the 1024 actors' rings (64 slots each)
    rs = g.RingSet(n, 64, device=dev)
    rng = np.random.default_rng(w["seed"])
    fi = t_(torch, dev, datagen.random_frames(rng, n * 7056).reshape(1, n, 84, 84))
    ei = torch.zeros((1, n), dtype=torch.uint8, device=dev)
    ai = torch.zeros((1, n), dtype=torch.int32, device=dev)
    ri = torch.zeros((1, n), dtype=torch.float32, device=dev)
    ins = lambda: g.gorila_replay_insert(ctx, rs, fi, ei, ai, ri)
    for _ in range(warmup):
        ins()
    ims = time_region(torch, ins, steps)
    ctx.check()
    ctx.close()
    ibytes = 2 * n * 7056 + n * (1 + 4 + 4) * 2
    flops = n * 2 * (MAC_CONV1 + MAC_CONV2 + MAC_CONV3 + MAC_FC1 + 512 * A)
    tf = flops / (ms * 1e-3) / 1e12
    return {"workload": "actor_n1024_a18_f32", "value": round(n / (ms * 1e-3), 1),
            "unit": "envs/s", "ms_per_call": round(ms, 4), "tflops": round(tf, 2),
            "pct_mfma_peak": round(100 * tf / FP32_MFMA_PEAK_TFLOPS, 2),
            "replay_insert": {"ms_per_call": round(ims, 4), "bytes": ibytes,
                              "gb_per_s": round(ibytes / (ims * 1e-3) / 1e9, 1)}}


def t_(torch, dev, a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def run_ring(torch, g, datagen, steps, warmup):
    """One-million-frame replay ring: the 256-index gather alone (bytes moved
    against HBM peak) and the batch-256 learner step reading the ring."""
    w = datagen.WORKLOADS["ring1m_gather_learner_b256_a18_f32"]
    B, A, cap = w["batch"], w["n_actions"], w["capacity"]
    rng = np.random.default_rng(w["seed"])
    r = datagen.ring_inputs(rng, cap, A)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    rep = g.Replay.ring(t(r.frames), t(r.ep_start), t(r.action), t(r.reward), r.head)
    del r
    idx = t(rng.integers(0, cap - 1, B).astype(np.int64))
    ctx = g.Context(B, A, device=dev)
    s = torch.empty((B, 4, 84, 84), dtype=torch.uint8, device=dev)
    s2, fmap = torch.empty_like(s), torch.empty((B, 2, 4), dtype=torch.int64, device=dev)
    a = torch.empty(B, dtype=torch.int32, device=dev)
    rr = torch.empty(B, dtype=torch.float32, device=dev)
    term = torch.empty(B, dtype=torch.uint8, device=dev)
    gather = lambda: g.gorila_gather(ctx, rep, idx, s, s2, fmap, a, rr, term)
    for _ in range(warmup):
        gather()
    ctx.check()
    # the call is launch-bound: time it eagerly and as 16 calls captured in
    # one HIP graph (the kernel rate without host-side launch overhead)
    gms_eager = time_region(torch, gather, steps)
    gr = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gr):
        for _ in range(16):
            gather()
    gr.replay()
    gms = time_region(torch, gr.replay, steps) / 16
    ctx.bind_stream()
    ctx.check()
    # algorithmic bytes: each distinct non-zero frame of s and s' read once
    # (they share up to three), both stacks written
    fm = fmap.cpu().numpy().reshape(B, 8)
    read = sum(len(set(row.tolist()) - {-1}) for row in fm) * 7056
    written = 2 * B * 28224
    gbs = (read + written) / (gms * 1e-3) / 1e9
    rng2 = np.random.default_rng(w["seed"] + 100)
    theta = t(datagen.he_normal_params(rng2, A).astype(np.float32))
    tgt = theta + 0.01 * torch.randn(theta.shape[0], device=dev, generator=torch.Generator(dev).manual_seed(5))
    grads = torch.empty(g.param_count(A), dtype=torch.float32, device=dev)
    loss = torch.empty(1, dtype=torch.float32, device=dev)
    step = lambda: g.gorila_learner_step(ctx, theta, tgt, A, rep, idx, 0.99, 1.0, grads, loss)
    for _ in range(warmup):
        step()
    ctx.check()
    lms = time_region(torch, step, steps)
    ctx.check()
    ctx.close()
    return {"workload": "ring1m_gather_learner_b256_a18_f32",
            "gather": {"ms_per_call": round(gms, 4), "ms_per_call_eager": round(gms_eager, 4),
                       "bytes": read + written,
                       "gb_per_s": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)},
            "learner": {"value": round(B / (lms * 1e-3), 1), "unit": "transitions/s",
                        "ms_per_step": round(lms, 4),
                        "note": "the step reads the ring in place (gather folded into conv1 staging)"}}


def run_ps(torch, g, datagen, steps, warmup):
    """Parameter-server apply of 16 learner gradients of the 18-action network
    (every gradient fresh and kept, so all 16 are applied), and the
    loss-statistics filter of 16 learners."""
    w = datagen.WORKLOADS["ps_apply_g16_a18_f32"]
    G, P = w["groups"], datagen.param_count(w["n_actions"])
    inp = datagen.ps_inputs(w["seed"], G, P)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    theta, accum, grads = t(inp.theta), t(inp.accum), t(inp.grads)
    ver = torch.zeros(G, dtype=torch.int64, device=dev)
    psv = torch.zeros(1, dtype=torch.int64, device=dev)
    applied = torch.empty(G, dtype=torch.uint8, device=dev)
    ctx = g.Context(1, w["n_actions"], device=dev)
    big = 1 << 62
    call = lambda: g.gorila_ps_apply(ctx, theta, accum, grads, ver, psv, big, 1e-4, 1e-3, applied)
    for _ in range(warmup):
        call()
    ctx.check()
    ms = time_region(torch, call, steps)
    assert int(applied.sum().item()) == G
    nbytes = P * 4 * (2 + G) + P * 4 * 2  # theta, accum and G gradients read; theta, accum written
    gbs = nbytes / (ms * 1e-3) / 1e9
    stats = torch.zeros((G, 3), dtype=torch.float64, device=dev)
    loss = t(datagen.loss_sequences(w["seed"], 1, G)[0])
    keep = torch.empty(G, dtype=torch.uint8, device=dev)
    filt = lambda: g.gorila_loss_filter(ctx, stats, loss, 0.05, 3.0, 10, keep)
    for _ in range(warmup):
        filt()
    fms = time_region(torch, filt, steps)
    ctx.check()
    ctx.close()
    return {"workload": "ps_apply_g16_a18_f32", "ms_per_call": round(ms, 4), "bytes": nbytes,
            "gb_per_s": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
            "loss_filter_ms_per_call": round(fms, 4)}


def cpu_baseline(datagen, B, A, seed, seconds):
    """The fp64 oracle (as it stands) running whole learner steps of the same
    batch-B workload on the host cores until `seconds` have passed."""
    import oracle
    inp = datagen.learner_inputs(seed, B, A)
    net = oracle.Net(n_actions=A)
    steps, t0 = 0, time.perf_counter()
    while True:
        oracle.learner_step(net, inp.theta, inp.theta_target, inp.s, inp.s2, inp.a, inp.r,
                            inp.term, inp.gamma, 1.0)
        steps += 1
        dt = time.perf_counter() - t0
        if dt >= seconds:
            break
    out = {"value": steps * B / dt, "unit": "transitions/s", "cores": oracle.num_threads(),
           "kind": "oracle", "host": host_cpu(),
           "sample": f"{steps} fp64 learner steps of the batch-{B} workload "
                     f"({steps * B} transitions, {dt:.1f} s)"}
    # one host thread, on the first 64 rows of the same workload (per-transition
    # cost does not depend on the batch size)
    nt = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        b1 = min(64, B)
        steps1, t0 = 0, time.perf_counter()
        while True:
            oracle.learner_step(net, inp.theta, inp.theta_target, inp.s[:b1], inp.s2[:b1],
                                inp.a[:b1], inp.r[:b1], inp.term[:b1], inp.gamma, 1.0)
            steps1 += 1
            dt1 = time.perf_counter() - t0
            if dt1 >= seconds / 2:
                break
    finally:
        oracle.set_num_threads(nt)
    out["single_thread"] = {"value": steps1 * b1 / dt1, "unit": "transitions/s", "cores": 1,
                            "sample": f"{steps1} fp64 learner steps on {b1} rows of the same "
                                      f"workload ({steps1 * b1} transitions, {dt1:.1f} s)"}
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batch", type=int, default=512)
    ap.add_argument("--actions", type=int, default=6)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-b32", action="store_true", help="skip the batch-32 companion line")
    ap.add_argument("--no-grouped", action="store_true",
                    help="skip the 16-replica bf16 grouped-step companion line")
    ap.add_argument("--no-actor", action="store_true", help="skip the actor-inference line")
    ap.add_argument("--no-two-learners", action="store_true",
                    help="skip the two-learners-on-two-streams lines")
    ap.add_argument("--no-ring", action="store_true",
                    help="skip the one-million-frame ring gather / learner line")
    ap.add_argument("--no-ps", action="store_true",
                    help="skip the parameter-server apply / loss-filter line")
    ap.add_argument("--only", choices=("actor", "grouped", "ring"), default=None,
                    help="only run that companion measurement and print its object "
                         "(profiles its kernels alone)")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes three times "
                         "(calibrates the HBM traffic counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1507_04296_amd as g
    from paper_1507_04296_amd import datagen
    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        src = torch.ones(args.copy_probe, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": args.copy_probe}), flush=True)
        return
    g.lib()  # fails loudly if the HIP library is missing
    if args.only == "actor":
        print(json.dumps({"actor": run_actor(torch, g, datagen, max(args.steps, 20), args.warmup)}),
              flush=True)
        return
    if args.only == "grouped":
        print(json.dumps({"grouped": run_grouped(torch, g, datagen, max(args.steps // 2, 5),
                                                 args.warmup)}), flush=True)
        return
    if args.only == "ring":
        print(json.dumps({"ring": run_ring(torch, g, datagen, max(args.steps, 20), args.warmup)}),
              flush=True)
        return

    B, A = args.batch, args.actions
    seed = datagen.SEED_BASE + 2
    r = run_learner(torch, g, datagen, B, A, seed, args.steps, args.warmup)
    fpt = step_flops_per_transition(A)
    step_tflops = B * fpt / (r["ms_per_step"] * 1e-3) / 1e12
    dom_flops = stage_flops(r["dominant"], B, A)
    dom_tflops = dom_flops / (r["dominant_ms"] * 1e-3) / 1e12
    stages = {k: {"ms": round(v[0] / max(v[1], 1), 4),
                  "tflops": round(stage_flops(k, B, A) / (v[0] / max(v[1], 1) * 1e-3) / 1e12, 2)}
              for k, v in r["prof"].items()}
    out = {
        "metric": "learner transitions/sec (DQN fwd+bwd) and % MFMA peak at batch 32/512",
        "value": round(B / (r["ms_per_step"] * 1e-3), 1),
        "unit": "transitions/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "settle_s": SETTLE_S,
        "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"learner_b{B}_a{A}_f32", "batch": B, "n_actions": A,
                   "replay": "stacked uint8 4x84x84", "gamma": 0.99, "clip_delta": 1.0,
                   "parallelism": "single GPU"},
        "tflops": round(step_tflops, 2),
        "pct_mfma_peak": round(100 * step_tflops / FP32_MFMA_PEAK_TFLOPS, 2),
        "flops_per_transition": fpt,
        "roofline": {"bound": "mfma", "kernel": r["dominant"], "achieved": round(dom_tflops, 2),
                     "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(dom_tflops / FP32_MFMA_PEAK_TFLOPS, 4),
                     "traffic": stored_traffic(r["dominant"], B, A),
                     "avg_launch_ms": round(r["dominant_ms"], 4),
                     "launches_timed": r["dominant_launches"],
                     "flops_per_launch": dom_flops},
        "step_ms_p10_p50_p90": r["pct"],
        "stages": stages,
    }
    # the same kernel's average from the committed rocprofv3 statistics (another
    # box and run: boxes differ by a few percent), beside the live figure
    prof_ms = stored_launch_ms(r["dominant"], B, A)
    if prof_ms is not None:
        out["roofline"]["profile"] = {
            "file": prof_ms[1], "avg_launch_ms": round(prof_ms[0], 4),
            "achieved": round(dom_flops / (prof_ms[0] * 1e-3) / 1e12, 2),
            "frac": round(dom_flops / (prof_ms[0] * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS, 4),
            "live_vs_profile": round(r["dominant_ms"] / prof_ms[0], 4)}
    if not args.no_b32:
        r32 = run_learner(torch, g, datagen, 32, 18, datagen.SEED_BASE + 0, max(args.steps, 50),
                          args.warmup, graph=True)
        t32 = 32 * step_flops_per_transition(18) / (r32["ms_per_step"] * 1e-3) / 1e12
        out["batch32"] = {"workload": "learner_b32_a18_f32",
                          "value": round(32 / (r32["ms_per_step"] * 1e-3), 1),
                          "ms_per_step": round(r32["ms_per_step"], 4), "tflops": round(t32, 3),
                          "pct_mfma_peak": round(100 * t32 / FP32_MFMA_PEAK_TFLOPS, 2),
                          "step_ms_p10_p50_p90": r32["pct"],
                          "hip_graph": {"ms_per_step": round(r32["graph_ms"], 4),
                                        "value": round(32 / (r32["graph_ms"] * 1e-3), 1)}}
    if not args.no_two_learners:
        out["two_learners"] = {
            "b512": run_two_learners(torch, g, datagen, B, A, seed, args.steps, args.warmup),
            "b32": run_two_learners(torch, g, datagen, 32, 18, datagen.SEED_BASE + 0,
                                    max(args.steps, 50), args.warmup)}
    if not args.no_grouped:
        out["grouped"] = run_grouped(torch, g, datagen, max(args.steps // 2, 5), args.warmup)
    if not args.no_actor:
        out["actor"] = run_actor(torch, g, datagen, max(args.steps, 20), args.warmup)
    if not args.no_ring:
        out["ring"] = run_ring(torch, g, datagen, max(args.steps, 20), args.warmup)
    if not args.no_ps:
        out["ps"] = run_ps(torch, g, datagen, max(args.steps, 20), args.warmup)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(datagen, B, A, seed, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
