#!/usr/bin/env python3
"""Benchmark of the per-layer MI hook step on one MI355X.

Default workload: the decode-shaped SAE hook step (d=4096, m=65536 latents,
TopK k=64, 256 decode tokens of which 128 requests subscribe, readback into
a 256-row ring): routing, SAE encode + top-k, ring compaction.  A step is
one full pass of that hook step, captured once as a HIP graph and replayed;
inputs are resident in HBM before timing starts.  The prefill-shaped SAE
step (8192 tokens, m=131072, k=32, plus 4 per-token and 4 pooled probes) is
timed in the same run and reported under "prefill".

The dictionaries (0.5 GiB and 1 GiB) are larger than the 256 MB
last-level cache, and each timed replay uses one of several copies in
rotation, so every replay streams its dictionary from HBM.

Prints one JSON line: hooked tokens/s per layer, the roofline fraction of
the dominant kernel (the encode GEMM, timed live with HIP events on the
stream it runs on) and the CPU oracle's rate on this host's cores.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--prefill-steps", type=int, default=20)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-decode", action="store_true",
                    help="profile only the prefill step (the JSON line then has no value)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle sample")
    ap.add_argument("--c5", action="store_true",
                    help="also time the 70B-shaped decode step (d=8192, T=R=512, 16 steering, "
                         "8 probe and 8 SAE clamp apps with 1 GiB dictionaries each)")
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


def time_replays(torch, rot, n):
    """Average ms per replay of `rot` over n replays, HIP events on the
    current stream (the stream the kernels run on)."""
    s = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(s)
    for _ in range(n):
        rot.replay()
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


def dictionary_copies(torch, W, min_bytes=1.5 * 2 ** 30):
    """W (a packed dictionary) and enough device copies of it that a
    rotation over them exceeds every cache."""
    n = max(STEPS_PER_GRAPH, int(np.ceil(min_bytes / W.nbytes)))
    return [W] + [W.clone() for _ in range(n - 1)]


def bench_workload(torch, px, step, sae_layer, sae_idx, steps, warmup, encode=True):
    """Times the full step and the encode GEMM (candidates stage)."""
    lay = step.layers[sae_layer]
    sae = lay.saes[sae_idx]
    copies = dictionary_copies(torch, sae.W_enc)

    def set_copy(W):
        sae.W_enc = W

    step.reset()
    step.run()   # eager run once (also checks the arguments)
    torch.cuda.synchronize()
    multi = MultiStep(torch, step.run, copies, set_copy, STEPS_PER_GRAPH, steps % STEPS_PER_GRAPH)
    for _ in range(max(1, warmup // STEPS_PER_GRAPH)):
        multi.full.replay()
    torch.cuda.synchronize()
    ms_step, per_run, sizes = time_step_runs(torch, multi, steps)
    stats = run_stats(per_run, sizes, step.wl.T_valid)
    ms_enc = encode_in_step(torch, step, copies, set_copy, steps) if encode else None
    set_copy(copies[0])
    return ms_step, ms_enc, stats


def encode_in_step(torch, step, copies, set_copy, n):
    """Average duration of the encode GEMM stage inside the step: n steps
    enqueued eagerly, back to back, with HIP events recorded on the step's
    stream right before and right after that stage (the step's other
    kernels run around it in the same order as in the captured step; the
    host enqueues far faster than the GPU runs a step, so the GPU sees the
    same back-to-back sequence)."""
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(n)]
    for i in range(3):
        set_copy(copies[i % len(copies)])
        step.run()
    torch.cuda.synchronize()
    for i, (e0, e1) in enumerate(pairs):
        set_copy(copies[i % len(copies)])
        step.run(marks=(e0.record, e1.record))
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in pairs) / n


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


def cpu_baseline_decode(wl, budget_s):
    """The oracle on this host's cores: one full decode SAE step is routing,
    the encode of every subscribed token and the ring compaction; the encode
    dominates, so a sample of subscribed tokens is encoded and the step time
    is scaled from it."""
    import oracle
    L = wl.layers[0]
    s = L.saes[0]
    t0 = time.perf_counter()
    tm, cnt, lists, err = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    t_route = time.perf_counter() - t0
    toks = lists[0, :cnt[0]]
    t0 = time.perf_counter()
    oracle.sae_encode(L.h, toks[:4], s.W_enc, s.b_enc, s.b_dec, s.k)
    per_tok = (time.perf_counter() - t0) / 4
    n = int(min(len(toks), max(4, budget_s / max(per_tok, 1e-9))))
    t0 = time.perf_counter()
    idx, val, _, _ = oracle.sae_encode(L.h, toks[:n], s.W_enc, s.b_enc, s.b_dec, s.k)
    t_enc = (time.perf_counter() - t0) / n * len(toks)
    idx_full = np.zeros((wl.T_max, s.k), np.int32)
    val_full = np.zeros((wl.T_max, s.k), np.uint16)
    t0 = time.perf_counter()
    oracle.compact([idx_full.view(np.uint8).reshape(wl.T_max, -1),
                    val_full.view(np.uint8).reshape(wl.T_max, -1)], tm, 0, wl.req, 0, 0,
                   np.zeros((s.ring_capacity, 16 + s.k * 6), np.uint8), 0)
    t_compact = time.perf_counter() - t0
    t_step = t_route + t_enc + t_compact
    return {"value": wl.T_valid / t_step, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{n} of {len(toks)} subscribed tokens encoded over all m latents "
                      f"(fp64), scaled to the full step; routing and compaction timed whole"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "the hook step runs on one GPU; sharding across GPUs is "
                                   "described, not implemented", "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    import synth
    import paper_2607_22595_amd as px
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
    if not args.no_decode:
        out, wl = run_decode(torch, px, synth, HookStep, args)
    if not args.no_decode:
        out["steer_probe"] = run_steer_probe(torch, synth, HookStep, args)
    if not args.no_prefill:
        out["prefill"] = run_prefill(torch, px, synth, HookStep, args)
    if args.c5:
        out["decode_70b"] = run_c5(torch, synth, HookStep, args)
    if not args.no_cpu_baseline and not args.no_decode:
        log("timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline_decode(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def run_decode(torch, px, synth, HookStep, args):
    log("generating the decode SAE workload")
    wl = synth.make("c3")
    step = HookStep(wl)
    log("timing the decode step")
    ms_step, ms_enc, stats = bench_workload(torch, px, step, 0, 0, args.steps, args.warmup)
    s = wl.layers[0].saes[0]
    n_sub = int(np.count_nonzero(wl.sub & 1))
    enc_bytes = s.m * wl.d * 2 + s.m * 4 + n_sub * wl.d * 2   # W_enc + folded bias + tokens
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
        "roofline": {"bound": "hbm", "kernel": "sae_stream_kernel (encode GEMM)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic("decode"),
                     "ms_per_launch": ms_enc, "algorithmic_bytes": enc_bytes,
                     "timing": "HIP events around the encode stage inside back-to-back steps"},
    }
    out["step_stats"] = stats
    log("measuring the HBM read ceiling")
    ceil = read_ceiling(torch, s.m * wl.d * 2)
    out["roofline"].update({
        "achievable_peak": ceil, "achievable_frac": achieved / ceil,
        "achievable_how": "nontemporal 16-byte read stream over 4 rotating buffers of the "
                          "dictionary's size, back-to-back launches (libxmix_ceiling)"})
    # "don't use, don't pay": the same captured step with no subscriber
    sub_saved = step.sub.clone()
    step.sub.zero_()
    ms_zero, _, _ = bench_workload(torch, px, step, 0, 0, args.steps, args.warmup, encode=False)
    step.sub.copy_(sub_saved)
    out["zero_mask_step_us"] = ms_zero * 1e3
    del step
    torch.cuda.empty_cache()
    return out, wl


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
        fn()
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(reps):
                fn()

        class One:
            def replay(self):
                g.replay()
        one = One()
        for _ in range(args.warmup):
            one.replay()
        return time_replays(torch, one, args.steps) * 1e3 / reps

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
    import time
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
    bits 0-3 steer, bits 4-7 probe), captured as one graph."""
    log("timing the 4-layer steering + probe decode step")
    wl = synth.make("c2")
    step = HookStep(wl)
    step.run()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step.run()

    class One:
        def replay(self):
            g.replay()
    one = One()
    for _ in range(args.warmup):
        one.replay()
    ms = time_replays(torch, one, args.steps)
    res = {"workload": "decode steering + probe step, 4 hooked layers, d=4096 T=R=256, "
                       "4 steering + 4 probe apps, subscriptions Bernoulli(0.3)",
           "us_per_step": ms * 1e3, "us_per_layer": ms * 1e3 / len(wl.layers),
           "value": wl.T_valid * len(wl.layers) / (ms * 1e-3), "unit": "hooked tokens/s per layer",
           "hbm_bytes": step.hbm_bytes()}
    res["conditional_us"] = time_conditional(torch, step, wl, args)
    log("timing parameter updates on the step graph")
    res["step_graph"] = time_step_graph(torch, step, args)
    del step
    torch.cuda.empty_cache()
    return res


def run_c5(torch, synth, HookStep, args):
    """The 70B-shaped decode step: steering, probes and eight SAE clamp apps,
    each encoding its subscribers over its own 1 GiB dictionary, captured as
    one graph.  The eight dictionaries (8 GiB) exceed every cache, so each
    replay streams them from HBM."""
    log("generating the 70B-shaped decode workload (8 dictionaries)")
    wl = synth.make("c5")
    step = HookStep(wl)
    step.run()
    torch.cuda.synchronize()
    # every replay starts from the same residual rows (steering and clamping
    # write them), restored by a device copy that is timed on its own too
    graphs = {}
    for name, body in (("step", lambda: (step.reset(), step.run())), ("restore", step.reset)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            body()
        graphs[name] = g

    class One:
        def __init__(self, g):
            self.g = g

        def replay(self):
            self.g.replay()
    log("timing the 70B-shaped decode step")
    times = {}
    for name, g in graphs.items():
        one = One(g)
        for _ in range(3):
            one.replay()
        times[name] = time_replays(torch, one, max(10, args.steps // 10))
    ms = times["step"] - times["restore"]
    nbytes = step.hbm_bytes()
    res = {"workload": "decode step d=8192 T=R=512: 16 steering, 8 probe and 8 SAE clamp apps "
                       "(m=65536, k=64, 4 clamped features each), subscriptions Bernoulli(0.2)",
           "ms_per_step": ms, "restore_ms": times["restore"],
           "value": wl.T_valid / (ms * 1e-3), "unit": "tokens/s",
           "algorithmic_bytes": nbytes, "achieved_GBps": nbytes / (ms * 1e-3) / 1e9,
           "frac_of_hbm_peak": nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    del graphs
    log("timing parameter updates on the 70B-shaped step graph")
    res["step_graph"] = time_step_graph(torch, step, args)
    del step
    torch.cuda.empty_cache()
    return res


def run_prefill(torch, px, synth, HookStep, args):
    log("generating the prefill workload")
    wl4 = synth.make("c4")
    step4 = HookStep(wl4)
    log("timing the prefill step")
    ms4, ms4_enc, stats4 = bench_workload(torch, px, step4, 0, 0, args.prefill_steps,
                                          max(2, args.warmup // 10))
    s4 = wl4.layers[0].saes[0]
    flops = 2.0 * wl4.T_valid * s4.m * wl4.d
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
                     "timing": "HIP events around the encode stage inside back-to-back steps",
                     "algorithmic_flops": flops,
                     "traffic": measured_traffic("prefill")},
        "step_stats": stats4}
    del step4
    torch.cuda.empty_cache()
    log("measuring the MFMA ceiling")
    ceil = mfma_ceiling(torch)
    res["roofline"].update({
        "achievable_peak": ceil, "achievable_frac": tf / ceil,
        "achievable_how": "32x32x16 bf16 MFMAs with register operands, 8 chains per wave, "
                          "4 waves per CU (libxmix_ceiling)"})
    return res


if __name__ == "__main__":
    main()
