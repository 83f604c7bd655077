#!/usr/bin/env python3
"""Benchmark of the per-layer MI hook step on one MI355X.

Headline (`value`): the decode-shaped SAE hook step (d=4096, m=65536
latents, TopK k=64, 256 decode tokens of which 128 requests subscribe,
readback into a 256-row ring): routing, SAE encode + top-k, ring readback.
A step is one full pass of that hook step, captured as a HIP graph and
replayed; inputs are resident in HBM before timing starts.  The dictionary
(0.5 GiB) is larger than the 256 MB last-level cache and each timed step
uses one of several copies in rotation, so every step streams it from HBM.

Timed in the same run, each in its own sub-record: the toy step (c1), the
4-layer steering + probe decode step (c2, hot and cold caches, conditional
filters, parameter updates on a step graph), the prefill step (c4), the
70B-shaped decode step with 8 SAE clamp apps (c5), the merge's repair path
on adversarial inputs, per-stage times of every step, and the CPU oracle on
this host's cores for every configuration.

Prints one JSON line: hooked tokens/s per layer, the roofline fraction of
the dominant kernel (the encode GEMM, timed live with HIP events on the
stream it runs on) and the CPU oracle's rate.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s
SETTLE_S = 0.3                  # untimed replays before the warmup steps


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--prefill-steps", type=int, default=20)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the decode steps (the JSON line then has no value)")
    ap.add_argument("--no-c5", action="store_true",
                    help="skip the 70B-shaped decode step (8 dictionaries of 1 GiB)")
    ap.add_argument("--no-repair", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run three device copies of 512 MiB, the known-size reference "
                         "for scaling HBM counter readings")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "sae_encode_hbm_traffic.md")
ENCODE_SOURCE = os.path.join(ROOT, "paper_2607_22595_amd", "csrc", "sae_encode.hip")


def measured_traffic(workload):
    """HBM bytes per launch of the encode GEMM from the committed rocprofv3
    counter summary (FETCH_SIZE and WRITE_SIZE, each scaled by what the same
    counter reads for a plain copy of known size), or None when the summary
    is missing or the kernel source changed since the counters were taken."""
    import hashlib
    try:
        text = open(TRAFFIC_FILE).read()
        src = hashlib.sha256(open(ENCODE_SOURCE, "rb").read()).hexdigest()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            fields[k.strip("`")] = v.strip().strip("`")
    if fields.get("source_sha256") != src:
        return None
    v = fields.get(f"{workload}_hbm_bytes_per_launch")
    return float(v) if v else None


# ------------------------------------------------------------------ timing

STEPS_PER_GRAPH = 4


class MultiStep:
    """One graph of `per_graph` consecutive steps (as consecutive hooked
    layers sit in one forward-pass graph), dictionary copies rotating from
    step to step, plus a graph of `rest` steps for a count that is not a
    multiple of it."""

    def __init__(self, torch, fn, copies, set_copy, per_graph, rest):
        def capture(n):
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(n):
                    set_copy(copies[i % len(copies)])
                    fn()
            return g
        self.per_graph = per_graph
        self.full = capture(per_graph)
        self.rest = capture(rest) if rest else None
        set_copy(copies[0])


def settle(torch, replay, seconds=SETTLE_S):
    """Untimed replays for `seconds`, so that the timed steps run at the
    device's steady clocks (generating the inputs leaves the GPU idle
    beforehand)."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n = 0
    while time.perf_counter() - t0 < seconds:
        replay()
        n += 1
        if n % 8 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    return n


def time_step_runs(torch, ms, n_steps, runs=7):
    """Exactly n_steps steps: n_steps // per_graph replays of the full graph
    and one of the rest graph, in `runs` consecutive runs with one HIP event
    between runs on the current stream (the stream the kernels run on).
    Returns the average ms per step and the per-run averages and sizes."""
    n_full = n_steps // ms.per_graph
    runs = max(1, min(runs, n_full)) if n_full else 1
    sizes = [n_full // runs + (1 if i < n_full % runs else 0) for i in range(runs)]
    s = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(runs + 1)]
    torch.cuda.synchronize()
    ev[0].record(s)
    steps = []
    for i, k in enumerate(sizes):
        for _ in range(k):
            ms.full.replay()
        n = k * ms.per_graph
        if i == runs - 1 and ms.rest is not None:
            ms.rest.replay()
            n += n_steps - n_full * ms.per_graph
        steps.append(n)
        ev[i + 1].record(s)
    ev[-1].synchronize()
    per_run = [ev[i].elapsed_time(ev[i + 1]) / steps[i] for i in range(runs)]
    return ev[0].elapsed_time(ev[-1]) / n_steps, per_run, steps


def time_replays(torch, replay, n):
    """Average ms per call of `replay` over n calls, HIP events on the
    current stream (the stream the kernels run on)."""
    s = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(s)
    for _ in range(n):
        replay()
    e1.record(s)
    e1.synchronize()
    return e0.elapsed_time(e1) / n


def run_stats(per_run, sizes, tokens_per_step, seed=0):
    """Median and p10/p90 of the per-run latency; the throughput over all
    runs (total tokens / total time, the harmonic mean of the per-run
    throughputs weighted by their replays) and a bootstrap 95 % interval of
    it over runs."""
    ms = np.asarray(per_run, np.float64)
    w = np.asarray(sizes, np.float64)
    thr = tokens_per_step * w.sum() / (ms * w).sum() * 1e3
    rng = np.random.default_rng(seed)
    boot = []
    for _ in range(2000):
        i = rng.integers(0, len(ms), len(ms))
        boot.append(tokens_per_step * w[i].sum() / (ms[i] * w[i]).sum() * 1e3)
    lo, hi = np.percentile(boot, [2.5, 97.5])
    return {"runs": len(ms), "steps_per_run": [int(x) for x in sizes],
            "steps_per_graph": STEPS_PER_GRAPH,
            "ms_median": float(np.median(ms)), "ms_p10": float(np.percentile(ms, 10)),
            "ms_p90": float(np.percentile(ms, 90)), "tokens_per_s": float(thr),
            "tokens_per_s_ci95": [float(lo), float(hi)]}


def stage_times(torch, step, n, before=None, warm=3):
    """Average time (us) of each stage of a hook step: n steps enqueued
    eagerly, back to back, with a HIP event recorded on the step's stream
    right before each stage and after the last (HookStep.run's `mark`).  A
    stage's time runs from its event to the next one: its kernels and the
    dispatch gap before them.  The host enqueues far faster than the GPU
    runs a step, so the GPU sees the same back-to-back sequence as in the
    captured step.  `before(i)` runs ahead of step i, outside every stage
    (dictionary rotation, restore copies)."""
    recs = []
    for i in range(n + warm):
        if before is not None:
            before(i)
        evs = []

        def mark(name, evs=evs):
            e = torch.cuda.Event(enable_timing=True)
            e.record()
            evs.append((name, e))
        step.run(mark=mark)
        if i >= warm:
            recs.append(evs)
    torch.cuda.synchronize()
    acc = {}
    for evs in recs:
        for (name, ea), (_, eb) in zip(evs[:-1], evs[1:]):
            acc.setdefault(name, []).append(ea.elapsed_time(eb) * 1e3)
    return {k: round(float(np.mean(v)), 3) for k, v in acc.items()}


def stage_times_graph(torch, step, n=10, before=None, rotate=None):
    """Per stage of a hook step: the GPU time (us) of one launch of that
    stage alone, from a graph of R back-to-back launches of it (the same
    arguments as in the step; the device state it reads is the one a full
    step left) replayed n times, divided by R.  R is 20 for stages under
    0.2 ms, else 1.  This is the time the stage takes inside a captured
    step, launch of its kernels in the graph included; unlike events
    between eager launches, it does not depend on the host's enqueue rate
    for short kernels.  `before()` runs ahead of the full step (restore
    copies).  rotate = (copies, set_copy): the encode stages' launches
    cycle through the dictionary copies (R at least their number), so that
    no launch finds its dictionary in a cache."""
    names = step.stage_names()
    if before is not None:
        before()
    step.run()
    torch.cuda.synchronize()
    out = {}
    for name in names:
        rot = rotate is not None and "encode" in name
        reps = len(rotate[0]) if rot else 1

        def launches():
            for i in range(reps):
                if rot:
                    rotate[1](rotate[0][i % len(rotate[0])])
                step.run(only=name)
            if rot:
                rotate[1](rotate[0][0])
        for _ in range(2):
            g = graph_of(torch, launches)
            g.replay()
            ms = time_replays(torch, g.replay, n) / reps
            del g
            if reps >= 20 or ms > 0.2:
                break
            reps = 20
        out[name] = round(ms * 1e3, 3)
    return out


def dictionary_copies(torch, W, min_bytes=1.5 * 2 ** 30):
    """W (a packed dictionary) and enough device copies of it that a
    rotation over them exceeds every cache."""
    n = max(STEPS_PER_GRAPH, int(np.ceil(min_bytes / W.nbytes)))
    return [W] + [W.clone() for _ in range(n - 1)]


def timed_sae_step(torch, step, steps, warmup, n_stage):
    """Times a step whose first layer holds one SAE app: the step graphs
    with the dictionary rotating over copies (settle, W warmup steps, then
    exactly `steps` timed steps), and the per-stage times."""
    sae = step.layers[0].saes[0]
    copies = dictionary_copies(torch, sae.W_enc)

    def set_copy(W):
        sae.W_enc = W

    step.reset()
    step.run()   # eager run once (also checks the arguments)
    torch.cuda.synchronize()
    multi = MultiStep(torch, step.run, copies, set_copy, STEPS_PER_GRAPH, steps % STEPS_PER_GRAPH)
    settle(torch, multi.full.replay)
    for _ in range(max(1, warmup // STEPS_PER_GRAPH)):
        multi.full.replay()
    torch.cuda.synchronize()
    ms_step, per_run, sizes = time_step_runs(torch, multi, steps)
    stats = run_stats(per_run, sizes, step.wl.T_valid)
    stages = stage_times(torch, step, n_stage,
                         before=lambda i: set_copy(copies[i % len(copies)]))
    set_copy(copies[0])
    stages["graph"] = stage_times_graph(torch, step, rotate=(copies, set_copy))
    return ms_step, stats, stages, multi


def read_ceiling(torch, nbytes, n_bufs=4, runs=7, per_run=20):
    """The device's measured HBM read ceiling: a plain stream of nontemporal
    16-byte loads (libxmix_ceiling) over `n_bufs` rotating buffers of the
    dictionary's size, back-to-back launches; median GB/s over the runs."""
    from paper_2607_22595_amd import ceiling
    bufs = [torch.empty(nbytes, dtype=torch.uint8, device="cuda") for _ in range(n_bufs)]
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for i in range(2 * n_bufs):
        ceiling.read(bufs[i % n_bufs], sink)
    rates = []
    for _ in range(runs):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(per_run):
            ceiling.read(bufs[i % n_bufs], sink)
        e1.record()
        e1.synchronize()
        rates.append(nbytes * per_run / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    del bufs
    torch.cuda.empty_cache()
    return float(np.median(rates))


def mfma_ceiling(torch, iters=4000, runs=7, per_run=3):
    """The device's measured bf16 MFMA ceiling (libxmix_ceiling): register
    operands only, one workgroup of four waves per CU; median TFLOP/s."""
    from paper_2607_22595_amd import ceiling
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    flops = ceiling.mfma(iters, sink)
    torch.cuda.synchronize()
    rates = []
    for _ in range(runs):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(per_run):
            ceiling.mfma(iters, sink)
        e1.record()
        e1.synchronize()
        rates.append(flops * per_run / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    return float(np.median(rates))


def graph_of(torch, fn):
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


# ----------------------------------------------------------- workloads

def run_decode(torch, synth, HookStep, args):
    log("generating the decode SAE workload (c3)")
    wl = synth.make("c3")
    step = HookStep(wl)
    log("timing the decode step")
    n_stage = max(200, args.steps)
    ms_step, stats, stages, multi = timed_sae_step(torch, step, args.steps, args.warmup, n_stage)
    s = wl.layers[0].saes[0]
    n_sub = int(np.count_nonzero(wl.sub & 1))
    enc_bytes = s.m * wl.d * 2 + s.m * 4 + n_sub * wl.d * 2   # W_enc + folded bias + tokens
    # the encode kernel's launch duration: graphs of back-to-back launches
    # (each on the next dictionary copy), the closest a HIP event gets to
    # the kernel's own duration; the eager figure adds the dispatch gaps
    ms_enc = stages["graph"]["L0/sae0/route+encode"] * 1e-3
    ms_enc_eager = stages["L0/sae0/route+encode"] * 1e-3
    achieved = enc_bytes / (ms_enc * 1e-3) / 1e9
    out = {
        "metric": "hooked tokens/sec per layer + % HBM/MFMA roofline (decode & prefill shapes)",
        "value": wl.T_valid / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; shapes of the paper's 8B-class served models)",
        "config": {"workload": "decode SAE hook step: route + encode/top-k + ring readback, "
                               "d=4096 m=65536 k=64 T=256 T_sub=128 ring=256",
                   "global_batch": wl.T_valid, "seq_len": 1, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": "sae_stream_kernel (encode GEMM, routing built "
                                               "in the same launch)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic("decode"),
                     "ms_per_launch": ms_enc, "algorithmic_bytes": enc_bytes,
                     "timing": "HIP events on the step's stream around graphs of back-to-back "
                               "launches of the encode stage, each launch on the next "
                               "dictionary copy",
                     "eager_ms_per_launch": ms_enc_eager, "eager_launches_timed": n_stage},
        "settle_s": SETTLE_S,
    }
    out["step_stats"] = stats
    out["stages_us"] = stages.pop("graph")
    out["stages_eager_us"] = stages
    log("measuring the HBM read ceiling")
    ceil = read_ceiling(torch, s.m * wl.d * 2)
    out["roofline"].update({
        "achievable_peak": ceil, "achievable_frac": achieved / ceil,
        "achievable_how": "nontemporal 16-byte read stream over 4 rotating buffers of the "
                          "dictionary's size, back-to-back launches (libxmix_ceiling)"})
    # "don't use, don't pay": the same captured steps with no subscriber
    sub_saved = step.sub.clone()
    step.sub.zero_()
    settle(torch, multi.full.replay, 0.1)
    ms_zero, _, _ = time_step_runs(torch, multi, max(args.steps, 100))
    step.sub.copy_(sub_saved)
    torch.cuda.synchronize()
    out["zero_mask_step_us"] = ms_zero * 1e3
    del multi, step
    torch.cuda.empty_cache()
    return out, wl


def run_toy(torch, synth, HookStep, args):
    """c1: 16 tokens of 4 requests, fp32, one steering and one probe app."""
    log("timing the toy step (c1)")
    wl = synth.make("c1")
    step = HookStep(wl)
    g = graph_of(torch, step.run)
    settle(torch, g.replay, 0.05)
    ms = time_replays(torch, g.replay, max(50, args.steps))
    res = {"workload": "toy step, 1 layer, fp32: d=256 T=16 R=4, 1 steering + 1 probe app "
                       "(routing built inside the fused probe + steering pass: one kernel)",
           "us_per_step": ms * 1e3,
           "value": wl.T_valid / (ms * 1e-3), "unit": "hooked tokens/s per layer",
           "note": "one graph launch per step: the graph's launch latency is most of it",
           "stages_us": stage_times_graph(torch, step)}
    del step
    return res, wl


def time_conditional(torch, step, wl, args):
    """Cost of the two conditional-write filters on the c2 batch: route build
    plus the filter, minus route build alone (each repeated 20 times inside
    one graph, so graph launch overhead drops out)."""
    import paper_2607_22595_amd as px
    import synth
    logit = step.layers[0].probes[0].logit[0]            # layer-0 probe, bit 4
    thr = torch.zeros(1, dtype=torch.float32, device="cuda")
    V = 128256
    ids = torch.from_numpy(synth.randint("bench/token_ids", wl.T_max, 0, V - 1)
                           .astype(np.int32)).cuda()
    vocab_bits = torch.zeros((V + 31) // 32, dtype=torch.int32, device="cuda")
    vocab_bits[::7] = -1                                  # a trigger set of ~1/7 of the ids

    def build():
        px.xmix_route_build(step.req, step.T_valid, step.sub, step.route, step.err)

    reps = 20

    def timed(fn):
        g = graph_of(torch, lambda: [fn() for _ in range(reps)])
        for _ in range(args.warmup):
            g.replay()
        return time_replays(torch, g.replay, args.steps) * 1e3 / reps

    # router-logit write on a Mixtral-shaped router (8 experts, bf16 logits),
    # bits 0-3 as four router apps; -inf offsets remove experts
    E = 8
    router_logits = torch.from_numpy(synth.normal_f32("bench/router_logits", (wl.T_max, E), 1.0)
                                     ).to(torch.bfloat16).cuda()
    off = synth.normal_f32("bench/router_offsets", (4, E), 1.0)
    off[synth.uniform01("bench/router_mask", 4 * E).reshape(4, E) < 0.2] = -np.inf
    off = torch.from_numpy(off).cuda()
    base = timed(build)
    gate = timed(lambda: (build(), px.xmix_route_gate(step.route, 1, logit, thr, signal_bit=4)))
    trig = timed(lambda: (build(), px.xmix_route_trigger(step.route, 2, ids, vocab_bits, V)))
    router = timed(lambda: (build(), px.xmix_router_write(router_logits, step.route, [0, 1, 2, 3],
                                                          off)))
    return {"route_build": base, "gate": gate - base, "trigger": trig - base,
            "router_write_8_experts": router - base}


def time_step_graph(torch, step, args):
    """Parameter updates on the library's own step graph of `step` (Sec. 4.3):
    per step, GPU time (events on the graph's stream) and host time to
    enqueue, for a plain launch; a launch after an in-memory update of alpha
    (one hipMemcpyAsync into the buffer the graph reads, from pinned host
    memory or from a preset device buffer); a launch after a kernel-node
    update that points every steering node at another alpha buffer; the
    zero-mask step (subscriptions buffer redirected to zeros); and a graph of
    one kernel that finds nothing to do, the floor of any graph launch."""
    import ctypes
    import paper_2607_22595_amd as px
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                   ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int
    stream = torch.cuda.Stream()
    step.reset()
    torch.cuda.synchronize()

    def record():
        # each replay first restores the residual rows (device copies), so
        # that steering and clamping do not drift over the replays
        with torch.cuda.stream(stream):
            step.reset()
        step.run(stream)
    g = px.Graph(record, stream)
    n = max(50, args.steps)

    def loop(fn):
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        t0 = time.perf_counter()
        for _ in range(n):
            fn()
        host = (time.perf_counter() - t0) / n * 1e6
        e1.record(stream)
        e1.synchronize()
        return {"gpu_us": e0.elapsed_time(e1) * 1e3 / n, "host_us": host}

    alpha0 = step.alpha
    alpha1 = alpha0.clone()
    pinned = alpha0.cpu().pin_memory()
    nbytes = alpha0.numel() * 4
    sptr = stream.cuda_stream
    res = {"kernel_nodes": g.kernel_nodes, "alpha_bytes": nbytes,
           "note": "every step graph replay includes the restore copies of the residual rows"}
    res["launch"] = loop(g.launch)

    rc = [0]

    def in_memory_h2d():
        rc[0] |= hip.hipMemcpyAsync(alpha0.data_ptr(), pinned.data_ptr(), nbytes, 1, sptr)
        g.launch()
    res["alpha_in_memory_h2d"] = loop(in_memory_h2d)
    preset = alpha0.clone()

    def in_memory_d2d():
        rc[0] |= hip.hipMemcpyAsync(alpha0.data_ptr(), preset.data_ptr(), nbytes, 3, sptr)
        g.launch()
    res["alpha_in_memory_d2d"] = loop(in_memory_d2d)
    if rc[0]:
        raise RuntimeError("hipMemcpyAsync failed in the parameter-update timing")
    cur = [alpha0, alpha1]
    updated = [0]

    def node_update():
        updated[0] = g.redirect(cur[0], cur[1])
        cur.reverse()
        g.launch()
    res["alpha_node_update"] = loop(node_update)
    res["alpha_node_update"]["args_per_update"] = updated[0]
    if cur[0] is not alpha0:
        g.redirect(cur[0], alpha0)
    zeros = torch.zeros_like(step.sub)
    g.redirect(step.sub, zeros)
    res["zero_mask"] = loop(g.launch)
    g.redirect(zeros, step.sub)
    # the floor: a graph of one library kernel that finds nothing to do (a
    # router write over a route no token subscribes to)
    rt = px.Route(1, 1)
    lg = torch.zeros((1, 1), dtype=torch.float32, device="cuda")
    off = torch.zeros((1, 1), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    eg = px.Graph(lambda: px.xmix_router_write(lg, rt, [0], off, stream), stream)
    res["empty_graph"] = loop(eg.launch)
    torch.cuda.synchronize()
    eg.close()
    g.close()
    step.reset()
    return res


def run_steer_probe(torch, synth, HookStep, args):
    """The 4-layer decode step of steering and probe apps (d=4096, T=R=256,
    bits 0-3 steer, bits 4-7 probe).  Hot: graphs of STEPS_PER_GRAPH
    consecutive steps (as the decode step's timing does) replayed back to
    back, so each step finds its rows in the caches as a layer does right
    after the model wrote them; also a graph of one step, whose replays each
    pay a graph launch.  Cold: before each timed one-step graph a 512 MiB
    write evicts the caches (outside the timed interval)."""
    log("timing the 4-layer steering + probe decode step (c2)")
    wl = synth.make("c2")
    step = HookStep(wl)
    g = graph_of(torch, step.run)

    def steps():
        for _ in range(STEPS_PER_GRAPH):
            step.run()
    gm = graph_of(torch, steps)
    settle(torch, gm.replay, 0.1)
    for _ in range(args.warmup):
        gm.replay()
    n_rep = max(1, args.steps // STEPS_PER_GRAPH)
    ms = time_replays(torch, gm.replay, n_rep) / STEPS_PER_GRAPH
    ms_single = time_replays(torch, g.replay, args.steps)
    flush = torch.empty(512 * 2 ** 20, dtype=torch.uint8, device="cuda")
    cold = []
    for _ in range(max(20, args.steps // 4)):
        flush.zero_()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        cold.append((e0, e1))
    torch.cuda.synchronize()
    ms_cold = float(np.mean([a.elapsed_time(b) for a, b in cold]))
    del flush
    res = {"workload": "decode steering + probe step, 4 hooked layers, d=4096 T=R=256, "
                       "4 steering + 4 probe apps, subscriptions Bernoulli(0.3)",
           "us_per_step": ms * 1e3, "us_per_layer": ms * 1e3 / len(wl.layers),
           "steps_per_graph": STEPS_PER_GRAPH,
           "one_step_graph_us_per_step": ms_single * 1e3,
           "cold_us_per_step": ms_cold * 1e3,
           "value": wl.T_valid * len(wl.layers) / (ms * 1e-3), "unit": "hooked tokens/s per layer",
           "hbm_bytes": step.hbm_bytes(),
           "stages_us": stage_times_graph(torch, step)}
    res["conditional_us"] = time_conditional(torch, step, wl, args)
    log("timing parameter updates on the step graph")
    res["step_graph"] = time_step_graph(torch, step, args)
    del step, g, gm
    torch.cuda.empty_cache()
    return res, wl


def run_c5(torch, synth, HookStep, args):
    """The 70B-shaped decode step: steering, probes and eight SAE clamp apps,
    each encoding its subscribers over its own 1 GiB dictionary, captured as
    one graph.  The eight dictionaries (8 GiB) exceed every cache, so each
    replay streams them from HBM."""
    log("generating the 70B-shaped decode workload (c5, 8 dictionaries)")
    wl = synth.make("c5")
    step = HookStep(wl)
    step.run()
    torch.cuda.synchronize()
    # every replay starts from the same residual rows (steering and clamping
    # write them), restored by a device copy that is timed on its own too
    graphs = {"step": graph_of(torch, lambda: (step.reset(), step.run())),
              "restore": graph_of(torch, step.reset)}
    log("timing the 70B-shaped decode step")
    settle(torch, graphs["step"].replay, 0.2)
    times = {}
    for name, g in graphs.items():
        for _ in range(3):
            g.replay()
        times[name] = time_replays(torch, g.replay, max(10, args.steps // 10))
    ms = times["step"] - times["restore"]
    nbytes = step.hbm_bytes()
    res = {"workload": "decode step d=8192 T=R=512: 16 steering, 8 probe and 8 SAE clamp apps "
                       "(m=65536, k=64, 4 clamped features each), subscriptions Bernoulli(0.2)",
           "ms_per_step": ms, "restore_ms": times["restore"],
           "value": wl.T_valid / (ms * 1e-3), "unit": "tokens/s",
           "algorithmic_bytes": nbytes, "achieved_GBps": nbytes / (ms * 1e-3) / 1e9,
           "frac_of_hbm_peak": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
           "stages_us": stage_times_graph(torch, step, n=3, before=step.reset)}
    del graphs
    log("timing parameter updates on the 70B-shaped step graph")
    res["step_graph"] = time_step_graph(torch, step, args)
    del step
    torch.cuda.empty_cache()
    return res, wl


def run_prefill(torch, synth, HookStep, args):
    log("generating the prefill workload (c4)")
    wl4 = synth.make("c4")
    step4 = HookStep(wl4)
    log("timing the prefill step")
    ms4, stats4, stages4, multi = timed_sae_step(torch, step4, args.prefill_steps,
                                                  max(2, args.warmup // 10), args.prefill_steps)
    s4 = wl4.layers[0].saes[0]
    flops = 2.0 * wl4.T_valid * s4.m * wl4.d
    ms4_enc = stages4["graph"]["L0/sae0/encode"] * 1e-3
    ms4_enc_eager = stages4["L0/sae0/encode"] * 1e-3
    tf = flops / (ms4_enc * 1e-3) / 1e12
    res = {
        "workload": "prefill hook step: route + 4 token probes + 4 pooled probes + SAE "
                    "encode/top-k, T=8192 R=16 d=4096 m=131072 k=32",
        "value": wl4.T_valid / (ms4 * 1e-3), "unit": "tokens/s", "ms_per_step": ms4,
        "steps": args.prefill_steps,
        "roofline": {"bound": "mfma",
                     "kernel": "sae_xstage_kernel + sae_gemm_kernel (encode GEMM)",
                     "achieved": tf, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tf / MFMA_BF16_PEAK_TFLOPS, "ms_per_launch": ms4_enc,
                     "timing": "HIP events on the step's stream around graphs of back-to-back "
                               "launches of the encode stage, each launch on the next "
                               "dictionary copy",
                     "eager_ms_per_launch": ms4_enc_eager,
                     "algorithmic_flops": flops,
                     "traffic": measured_traffic("prefill")},
        "step_stats": stats4, "stages_us": stages4.pop("graph"), "stages_eager_us": stages4}
    del multi, step4
    torch.cuda.empty_cache()
    log("measuring the MFMA ceiling")
    ceil = mfma_ceiling(torch)
    res["roofline"].update({
        "achievable_peak": ceil, "achievable_frac": tf / ceil,
        "achievable_how": "32x32x16 bf16 MFMAs with register operands, 8 chains per wave, "
                          "4 waves per CU (libxmix_ceiling)"})
    return res, wl4


# ------------------------------------------------- repair path, worst cases

def _strong_latents(synth, wl, scale=60.0):
    """Every subscribed token's row moved along three dictionary rows, so
    that those latents stand far above the token's others (as clamping
    features high leaves them)."""
    s = wl.layers[0].saes[0]
    h = synth.bf16_bits_to_f32(wl.layers[0].h).astype(np.float64)
    T = wl.T_max
    picks = synth.randint("bench/strong_latents", 3 * T, 0, s.m - 1).reshape(T, 3)
    for t in range(T):
        for j in picks[t]:
            w = synth.bf16_bits_to_f32(s.W_enc[j]).astype(np.float64)
            h[t] += scale * w / np.dot(w, w)
    u = h.astype(np.float32).view(np.uint32).astype(np.uint64)
    wl.layers[0].h = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)  # to bf16, RNE


def _tied_slices(wl, n_tied):
    """n_tied 256-latent slices whose pre-activations are all exactly 40:
    zero dictionary rows with bias 40, far above every other latent.  No
    threshold splits a tie, so those slices emit nothing and the merge must
    recompute them."""
    s = wl.layers[0].saes[0]
    n_mt = s.m // 256
    slices = np.arange(n_mt) if n_tied >= n_mt else 1 + (n_mt // n_tied) * np.arange(n_tied)
    W, b = s.W_enc.copy(), s.b_enc.copy()
    for sl in slices:
        W[256 * sl:256 * (sl + 1)] = 0
        b[256 * sl:256 * (sl + 1)] = 0x4220  # 40.0
    s.W_enc, s.b_enc = W, b


def _tied_candidates(synth, wl, rows=8):
    """In every 256-latent slice, `rows` identical dictionary rows along one
    direction the tokens share (zero bias), so that every slice emits that
    many candidates of exactly the same value far above the rest: with
    m=131072 a token's candidates overflow the merge's pool with ties."""
    s = wl.layers[0].saes[0]
    d = wl.d
    u = synth.bf16_bits_to_f32(synth.normal_bf16("bench/tied_pool/u", (d,), 1.0)).astype(np.float64)
    u /= np.linalg.norm(u)
    row = (10.0 / np.sqrt(d)) * u
    W, b = s.W_enc.copy(), s.b_enc.copy()
    tied = (np.arange(s.m) % 256) < rows
    W[tied] = _to_bf16(row)[None, :]
    b[tied] = 0
    s.W_enc, s.b_enc = W, b
    h = synth.bf16_bits_to_f32(wl.layers[0].h).astype(np.float64) + 3.0 * np.sqrt(d) * u[None, :]
    wl.layers[0].h = _to_bf16(h)


def _heavy_tailed(torch, synth, wl, alpha=1.5, cap=200.0):
    """Dictionary rows scaled by Pareto(alpha) factors (capped): a token's
    pre-activations over the latents become a scale mixture of normals with
    a power-law tail, which the first threshold guess (a slice's mean and
    stdev) misjudges: slices with a large factor overshoot the window and
    refine, the others keep few candidates."""
    s = wl.layers[0].saes[0]
    u = synth.uniform01("bench/heavy/scale", s.m)
    f = np.minimum((1.0 - u) ** (-1.0 / alpha), cap)
    W = s.W_enc.reshape(s.m, -1).copy()
    fs = torch.from_numpy(f.astype(np.float32))
    for r0 in range(0, s.m, 8192):  # in row blocks, to bound host memory
        blk = torch.from_numpy(W[r0:r0 + 8192].view(np.int16)).view(torch.bfloat16)
        # bf16 x fp32 is exact in fp32's 24 bits; one RNE rounding to bf16
        out = (blk.float() * fs[r0:r0 + 8192, None]).to(torch.bfloat16)
        W[r0:r0 + 8192] = out.view(torch.int16).numpy().view(np.uint16)
    s.W_enc = W.reshape(s.W_enc.shape)


def _to_bf16(x):
    u = np.asarray(x, np.float64).astype(np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)  # RNE


def run_repair(torch, synth, HookStep, args):
    """The merge's repair path on inputs built to defeat the candidate
    thresholds, at the decode SAE shape (c3) and with the prefill GEMM
    (1100 token slots, d=4096, m=131072, k=32): per case the encode and
    merge stage times of the step."""
    log("timing the repair path on adversarial inputs")
    cases = [("c3 plain", {}, None, 10),
             ("c3 strong latents (3 per token)", {}, "strong", 10),
             ("c3 10 tied slices", {}, 10, 10),
             ("c3 20 tied slices", {}, 20, 5),
             ("c3 every slice tied", {}, 256, 3),
             ("c3 heavy-tailed rows (Pareto 1.5 scales)", {}, "heavy", 10),
             ("prefill GEMM, 1100 tokens, strong latents", {"T": 1100, "n_sub": 1100,
                                                            "m": 131072, "k": 32}, "strong", 5),
             ("prefill GEMM, 1100 tokens, 10 tied slices", {"T": 1100, "n_sub": 1100,
                                                            "m": 131072, "k": 32}, 10, 5),
             ("prefill GEMM, 1100 tokens, every slice tied", {"T": 1100, "n_sub": 1100,
                                                              "m": 131072, "k": 32}, 512, 3),
             ("prefill GEMM, 1100 tokens, heavy-tailed rows (Pareto 1.5 scales)",
              {"T": 1100, "n_sub": 1100, "m": 131072, "k": 32}, "heavy", 5),
             ("prefill GEMM, 1100 tokens, 4096 tied candidates per token",
              {"T": 1100, "n_sub": 1100, "m": 131072, "k": 32, "n_outliers": 0}, "tied_pool", 3)]
    res = {}
    for name, kw, kind, n in cases:
        wl = synth.make("c3", ring_capacity=0, **kw)
        if kind == "strong":
            _strong_latents(synth, wl)
        elif kind == "tied_pool":
            _tied_candidates(synth, wl)
        elif kind == "heavy":
            _heavy_tailed(torch, synth, wl)
        elif kind is not None:
            _tied_slices(wl, kind)
        step = HookStep(wl)
        st = stage_times(torch, step, n, warm=1)
        enc = next(v for k, v in st.items() if k.endswith("encode"))
        res[name] = {"encode_us": enc, "merge_us": st["L0/sae0/merge"],
                     "tokens": int(np.count_nonzero(wl.sub & 1))}
        del step
        torch.cuda.empty_cache()
    return res


# ------------------------------------------------------------ CPU oracle

def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _timed(fn):
    t0 = time.perf_counter()
    fn()
    return time.perf_counter() - t0


def _encode_rate(oracle, L, s, toks, n):
    """Seconds per token of the oracle's encode over a sample of n tokens."""
    n = max(1, min(n, len(toks)))
    return _timed(lambda: oracle.sae_encode(L.h, toks[:n], s.W_enc, s.b_enc, s.b_dec, s.k)) / n


def _cpu_config(oracle, name, wl, n_all, n_one):
    """One configuration's oracle step on the host: the parts that are cheap
    are timed whole, the SAE encodes on token samples (n_all tokens with all
    threads, n_one single-threaded) and scaled to the full step.  Returns
    (seconds all-core, seconds single-thread, sample description)."""
    t = {}
    for label, threads, n_enc in (("all", oracle_threads(oracle), n_all), ("one", 1, n_one)):
        oracle.set_num_threads(threads)
        total = 0.0
        t0 = time.perf_counter()
        tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
        total += time.perf_counter() - t0
        for L in wl.layers:
            if L.steer:
                bits = [s.bit for s in L.steer]
                v = np.stack([s.v for s in L.steer])
                total += _timed(lambda: oracle.steer(L.h, tm, wl.req, v, bits, wl.alpha))
            for mode in ("token", "mean"):
                ps = [p for p in L.probes if p.mode == mode]
                if not ps:
                    continue
                w = np.stack([p.w for p in ps])
                b = np.array([p.b for p in ps], np.float32)
                bits = [p.bit for p in ps]
                if mode == "token":
                    total += _timed(lambda: oracle.probe_token(L.h, tm, w, b, bits))
                else:
                    total += _timed(lambda: oracle.probe_mean(L.h, tm, w, b, bits,
                                                              wl.cu_seqlens))
            for s in L.saes:
                toks = lists[s.bit, :cnt[s.bit]]
                if len(toks) == 0:
                    continue
                total += _encode_rate(oracle, L, s, toks, n_enc) * len(toks)
                if s.W_dec is not None:
                    idx = np.zeros((wl.T_max, s.k), np.int32)
                    val = np.zeros((wl.T_max, s.k), np.uint16)
                    total += _timed(lambda: oracle.clamp_decode(L.h, tm, s.bit, idx, val,
                                                                s.W_dec, s.clamp_ids,
                                                                s.clamp_vals))
                if s.ring_capacity:
                    idx = np.zeros((wl.T_max, s.k), np.int32)
                    val = np.zeros((wl.T_max, s.k), np.uint16)
                    slots = np.zeros((s.ring_capacity, 16 + 6 * s.k), np.uint8)
                    total += _timed(lambda: oracle.compact(
                        [idx.view(np.uint8).reshape(wl.T_max, -1),
                         val.view(np.uint8).reshape(wl.T_max, -1)], tm, s.bit, wl.req, 0,
                        s.bit, slots, 0))
        t[label] = total
    oracle.set_num_threads(oracle_threads(oracle))
    n_sae = sum(len(L.saes) for L in wl.layers)
    sample = ("whole step" if n_sae == 0 else
              f"whole step except the SAE encodes: {n_all} tokens per SAE app with all "
              f"threads, {n_one} single-threaded, each over all m latents, scaled to every "
              f"subscribed token")
    return t["all"], t["one"], sample


_THREADS = []


def oracle_threads(oracle):
    if not _THREADS:
        _THREADS.append(oracle.num_threads())
    return _THREADS[0]


def cpu_baseline(wls):
    """The CPU oracle (plain fp64 C, OpenMP over tokens) on this host: per
    configuration, tokens per second per hooked layer with all threads and
    with one thread.  The headline figure is the decode SAE step (c3)."""
    import oracle
    threads = oracle_threads(oracle)
    plan = {"c1": (0, 0), "c2": (0, 0), "c3": (128, 6), "c4": (48, 2), "c5": (8, 1)}
    per = {}
    for name, wl in wls.items():
        if wl is None:
            continue
        n_all, n_one = plan[name]
        log(f"timing the CPU oracle on {name}")
        t_all, t_one, sample = _cpu_config(oracle, name, wl, n_all, n_one)
        layers = len(wl.layers)
        per[name] = {"tokens_per_s_all_threads": wl.T_valid * layers / t_all,
                     "tokens_per_s_single_thread": wl.T_valid * layers / t_one,
                     "step_s_all_threads": t_all, "step_s_single_thread": t_one,
                     "single_thread": "measured" if name in ("c1", "c2") else
                     "extrapolated from the sample",
                     "sample": sample}
    head = per.get("c3") or next(iter(per.values()))
    return {"value": head["tokens_per_s_all_threads"], "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": "decode SAE step (c3): " + head["sample"],
            "cpu_model": _cpu_model(), "nproc": os.cpu_count(), "per_config": per}


# ------------------------------------------------------------------ main

def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the hook step runs on one GPU; sharding across GPUs is "
                                   "described, not implemented", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import synth
    from paper_2607_22595_amd.hookstep import HookStep

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        src = torch.empty(512 * 2 ** 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    out = {}
    wls = {}
    if not args.no_decode:
        out, wls["c3"] = run_decode(torch, synth, HookStep, args)
        out["steer_probe"], wls["c2"] = run_steer_probe(torch, synth, HookStep, args)
        out["toy"], wls["c1"] = run_toy(torch, synth, HookStep, args)
    if not args.no_prefill:
        out["prefill"], wls["c4"] = run_prefill(torch, synth, HookStep, args)
    if not args.no_decode and not args.no_c5:
        out["decode_70b"], wls["c5"] = run_c5(torch, synth, HookStep, args)
    if not args.no_repair:
        out["repair"] = run_repair(torch, synth, HookStep, args)
    if not args.no_cpu_baseline and wls:
        out["cpu_baseline"] = cpu_baseline(wls)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
