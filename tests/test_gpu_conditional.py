"""Conditional writes on the GPU: the routing filters against the oracle
(bit-exact), and the two app shapes they serve, end to end:
  - activation-driven (a probe at one layer gates steering at a later one,
    as in conditional refusal);
  - token-driven (steering only on tokens whose id is in a trigger list).
The gate decision is taken on the GPU's own fp32 probe logits on both sides
(stage isolation), so a logit that sits on the threshold cannot flip it."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_steer, torch_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def px():
    import paper_2607_22595_amd as m
    return m


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a).view(np.int32))).cuda()


def dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def gpu_route(px, req, T_valid, sub, n_apps):
    rt = px.Route(len(req), n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_build(dev_i32(req), torch.tensor([T_valid], dtype=torch.int32, device="cuda"),
                        dev_i32(np.asarray(sub, np.uint32)), rt, err)
    return rt


def route_host(rt):
    torch.cuda.synchronize()
    return (rt.tok_mask.cpu().numpy().view(np.uint32), rt.app_count.cpu().numpy(),
            rt.app_tokens.cpu().numpy())


def assert_route_equal(got, ref):
    assert np.array_equal(got[0], ref[0])
    assert np.array_equal(got[1], ref[1])
    assert np.array_equal(got[2], ref[2])


def _random_route(seed, T=3000, R=40, n_apps=6):
    rng = np.random.default_rng(seed)
    req = rng.integers(-1, R, T).astype(np.int32)
    sub = rng.integers(0, 1 << n_apps, R).astype(np.uint32)
    T_valid = T - int(rng.integers(0, 50))
    return rng, req, sub, T_valid, n_apps


@pytest.mark.parametrize("seed", range(4))
def test_gate_per_token_bit_exact(px, seed):
    rng, req, sub, T_valid, n_apps = _random_route(seed)
    T = len(req)
    rt = gpu_route(px, req, T_valid, sub, n_apps)
    sig = rng.normal(size=T).astype(np.float32)
    sig[rng.integers(0, T, 40)] = np.nan
    thr = np.float32(rng.normal() * 0.5)
    app, sbit = 1, (4 if seed % 2 else -1)
    before = route_host(rt)
    px.xmix_route_gate(rt, app, torch.from_numpy(sig).cuda(),
                       torch.tensor([thr], dtype=torch.float32, device="cuda"), signal_bit=sbit)
    ref = oracle.route_gate(*before, app, sig, float(thr), signal_bit=sbit)
    assert_route_equal(route_host(rt), ref)


@pytest.mark.parametrize("seed", range(2))
def test_gate_per_request_bit_exact(px, seed):
    rng, req, sub, T_valid, n_apps = _random_route(10 + seed)
    R = len(sub)
    rt = gpu_route(px, req, T_valid, sub, n_apps)
    sig = rng.normal(size=R).astype(np.float32)
    before = route_host(rt)
    px.xmix_route_gate(rt, 3, torch.from_numpy(sig).cuda(),
                       torch.zeros(1, dtype=torch.float32, device="cuda"), req_of_token=dev_i32(req))
    assert_route_equal(route_host(rt), oracle.route_gate(*before, 3, sig, 0.0, req=req))


@pytest.mark.parametrize("seed", range(3))
def test_trigger_bit_exact(px, seed):
    rng, req, sub, T_valid, n_apps = _random_route(20 + seed)
    T = len(req)
    V = 32000
    ids = rng.integers(-3, V + 3, T).astype(np.int32)
    trig = rng.choice(V, 1600, replace=False)
    bits = np.zeros((V + 31) // 32, np.uint32)
    np.bitwise_or.at(bits, trig >> 5, (np.uint32(1) << (trig & 31).astype(np.uint32)))
    ids[rng.integers(0, T, 200)] = trig[rng.integers(0, trig.size, 200)]  # make hits common
    rt = gpu_route(px, req, T_valid, sub, n_apps)
    before = route_host(rt)
    px.xmix_route_trigger(rt, 2, dev_i32(ids), dev_i32(bits), V)
    assert_route_equal(route_host(rt), oracle.route_trigger(*before, 2, ids, bits, V))


def test_gate_empty_and_full(px):
    rng, req, sub, T_valid, n_apps = _random_route(30)
    T = len(req)
    for thr, expect_all in ((-np.inf, True), (np.inf, False)):
        rt = gpu_route(px, req, T_valid, sub, n_apps)
        before = route_host(rt)
        px.xmix_route_gate(rt, 0, torch.zeros(T, dtype=torch.float32, device="cuda"),
                           torch.tensor([thr], dtype=torch.float32, device="cuda"))
        tm, cnt, lists = route_host(rt)
        assert cnt[0] == (before[1][0] if expect_all else 0)
        assert np.array_equal(lists[1:], before[2][1:])


def _two_layer_workload():
    # layer 0: probe app (bit 4); layer 1: steering apps (bits 0-3); the
    # steering app on bit 1 is conditional on the layer-0 probe
    return synth.make("c2", n_layers=2, T=300)


def test_activation_gated_steering_end_to_end(px):
    wl = _two_layer_workload()
    L0, L1 = wl.layers
    probe = [p for p in L0.probes if p.bit == 4][0]
    rt = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    # layer 0 probe (token mode) into a persistent signal row
    h0 = dev_bits(L0.h)
    logit = torch.full((1, wl.T_max), float("nan"), device="cuda")
    score = torch.full((1, wl.T_max), float("nan"), device="cuda")
    px.xmix_probe_score(h0, rt, dev_bits(probe.w[None]), torch.tensor([probe.b], device="cuda"),
                        [4], px.XMIX_PROBE_TOKEN, logit, score)
    before = route_host(rt)
    thr = torch.tensor([0.0], device="cuda")
    px.xmix_route_gate(rt, 1, logit[0], thr, signal_bit=4)
    # layer 1 steering with the gated route
    bits = [s.bit for s in L1.steer]
    v = np.stack([s.v for s in L1.steer])
    h1 = dev_bits(L1.h)
    px.xmix_steer_apply(h1, rt, dev_i32(wl.req), dev_bits(v), bits, torch.from_numpy(wl.alpha).cuda())
    torch.cuda.synchronize()
    # oracle chain on the GPU's own logits
    lg = logit[0].cpu().numpy()
    tm_g, _, _ = oracle.route_gate(*before, 1, lg, 0.0, signal_bit=4)
    assert np.array_equal(route_host(rt)[0], tm_g)
    ref = oracle.steer(L1.h, tm_g, wl.req, v, bits, wl.alpha)
    rows = (tm_g & np.uint32(sum(1 << b for b in bits))) != 0
    check_steer(torch_bits(h1), ref, L1.h, rows, True)
    # the gate removed some tokens and kept some
    had = (before[0] >> 1) & 1
    kept = (tm_g >> 1) & 1
    assert kept.sum() > 0 and kept.sum() < had.sum()


def test_token_triggered_steering_end_to_end(px):
    wl = _two_layer_workload()
    L1 = wl.layers[1]
    V = 50000
    ids = synth.randint("c2/token_ids", wl.T_max, 0, V - 1).astype(np.int32)
    trig = np.unique(ids[synth.permutation("c2/trigger_pick", wl.T_max)[:30]])
    bits_v = np.zeros((V + 31) // 32, np.uint32)
    np.bitwise_or.at(bits_v, trig >> 5, (np.uint32(1) << (trig & 31).astype(np.uint32)))
    rt = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    before = route_host(rt)
    px.xmix_route_trigger(rt, 2, dev_i32(ids), dev_i32(bits_v), V)
    bits = [s.bit for s in L1.steer]
    v = np.stack([s.v for s in L1.steer])
    h1 = dev_bits(L1.h)
    px.xmix_steer_apply(h1, rt, dev_i32(wl.req), dev_bits(v), bits, torch.from_numpy(wl.alpha).cuda())
    torch.cuda.synchronize()
    tm_t, _, _ = oracle.route_trigger(*before, 2, ids, bits_v, V)
    assert np.array_equal(route_host(rt)[0], tm_t)
    ref = oracle.steer(L1.h, tm_t, wl.req, v, bits, wl.alpha)
    rows = (tm_t & np.uint32(sum(1 << b for b in bits))) != 0
    check_steer(torch_bits(h1), ref, L1.h, rows, True)


def test_gate_in_graph_with_new_threshold(px):
    """Captured once; the threshold changes in device memory between replays."""
    rng, req, sub, T_valid, n_apps = _random_route(40, T=2000)
    T = len(req)
    rt = px.Route(T, n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    req_d, sub_d = dev_i32(req), dev_i32(sub)
    tv = torch.tensor([T_valid], dtype=torch.int32, device="cuda")
    sig = torch.from_numpy(rng.normal(size=T).astype(np.float32)).cuda()
    thr = torch.zeros(1, dtype=torch.float32, device="cuda")

    def step():
        px.xmix_route_build(req_d, tv, sub_d, rt, err)
        px.xmix_route_gate(rt, 5, sig, thr)

    step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    tm0, cnt0, lists0, _ = oracle.route(req, T_valid, sub, n_apps)
    for t in (0.0, 0.7, -0.3, 0.0):
        thr.fill_(t)
        g.replay()
        ref = oracle.route_gate(tm0, cnt0, lists0, 5, sig.cpu().numpy(), t)
        assert_route_equal(route_host(rt), ref)
