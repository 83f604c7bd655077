"""Router-logit write (mixture-of-experts expert (de)activation) on the GPU
against the oracle, bit-exact: both sides add the subscribed apps' offsets
in app order in fp64 and round once to the logits' storage type.  Inputs
are seeded; offsets mix finite values, -inf (expert removed) and large
positive values (expert forced)."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def px():
    import paper_2607_22595_amd as m
    return m


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a).view(np.int32))).cuda()


def gpu_route(px, req, T_valid, sub, n_apps):
    rt = px.Route(len(req), n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_build(dev_i32(req), torch.tensor([T_valid], dtype=torch.int32, device="cuda"),
                        dev_i32(np.asarray(sub, np.uint32)), rt, err)
    return rt


def host_mask(rt):
    torch.cuda.synchronize()
    return rt.tok_mask.cpu().numpy().view(np.uint32)


def make_logits(rng, T, E, dtype):
    x = rng.normal(0.0, 2.0, (T, E)).astype(np.float32)
    t = torch.from_numpy(x)
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
        return t.cuda(), t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.cuda(), x.copy()


def make_offsets(rng, n, E):
    off = rng.normal(0.0, 1.5, (n, E)).astype(np.float32)
    off[rng.random((n, E)) < 0.15] = -np.inf
    off[rng.random((n, E)) < 0.05] = 1e4
    return off


def host_bits(t):
    a = t.detach().cpu()
    if a.dtype == torch.bfloat16:
        return a.view(torch.int16).numpy().view(np.uint16)
    return a.numpy().view(np.uint32)


def as_bits(a):
    return a.view(np.uint16) if a.dtype == np.uint16 else a.view(np.uint32)


@pytest.mark.parametrize("E,dtype,T", [(8, "bf16", 300), (8, "f32", 77), (64, "bf16", 1025),
                                       (160, "f32", 513)])
def test_router_write_bit_exact(px, E, dtype, T):
    rng = np.random.default_rng(E * 7 + T)
    R, n_apps = 37, 6
    req = rng.integers(-1, R, T).astype(np.int32)
    sub = rng.integers(0, 1 << n_apps, R).astype(np.uint32)
    T_valid = T - 5
    rt = gpu_route(px, req, T_valid, sub, n_apps)
    bits = [4, 1, 3]
    off = make_offsets(rng, len(bits), E)
    lg, lg_host = make_logits(rng, T, E, dtype)
    px.xmix_router_write(lg, rt, bits, torch.from_numpy(off).cuda())
    ref = oracle.router_write(lg_host, host_mask(rt), bits, off)
    assert np.array_equal(host_bits(lg), as_bits(ref))


def test_router_write_masks_and_forces_experts(px):
    """Mixtral-shaped (8 experts, top-2): app 0 removes expert 2, app 1
    forces expert 6; the top-2 of a token then follows its subscriptions."""
    rng = np.random.default_rng(5)
    T, E = 256, 8
    req = np.arange(T, dtype=np.int32)
    sub = rng.integers(0, 4, T).astype(np.uint32)
    rt = gpu_route(px, req, T, sub, 2)
    off = np.zeros((2, E), np.float32)
    off[0, 2] = -np.inf
    off[1, 6] = 1e4
    lg, lg_host = make_logits(rng, T, E, "bf16")
    px.xmix_router_write(lg, rt, [0, 1], torch.from_numpy(off).cuda())
    out = lg.float().cpu().numpy()
    ref = oracle.router_write(lg_host, host_mask(rt), [0, 1], off)
    assert np.array_equal(host_bits(lg), ref)
    for t in range(T):
        top2 = set(np.argsort(-out[t], kind="stable")[:2].tolist())
        if sub[t] & 1:
            assert out[t, 2] == -np.inf and 2 not in top2
        if sub[t] & 2:
            assert 6 in top2


def test_router_write_no_subscribers_leaves_logits(px):
    rng = np.random.default_rng(6)
    T, E = 100, 8
    rt = gpu_route(px, np.arange(T, dtype=np.int32), T, np.zeros(T, np.uint32), 3)
    lg, lg_host = make_logits(rng, T, E, "bf16")
    px.xmix_router_write(lg, rt, [0, 1, 2], torch.from_numpy(make_offsets(rng, 3, E)).cuda())
    assert np.array_equal(host_bits(lg), lg_host)


def test_router_write_gated_by_probe(px):
    """Conditional form: a probe's logit gates the router app per token
    (xmix_route_gate), then the write applies only to the tokens that pass.
    The gate decision uses the GPU's own probe logits on both sides."""
    rng = np.random.default_rng(7)
    T, d, E = 300, 256, 8
    req = np.arange(T, dtype=np.int32)
    sub = np.full(T, 0b11, np.uint32)          # bit 0: probe, bit 1: router app
    rt = gpu_route(px, req, T, sub, 2)
    h = torch.from_numpy(rng.normal(0, 1, (T, d)).astype(np.float32)).to(torch.bfloat16).cuda()
    w = torch.from_numpy(rng.normal(0, d ** -0.5, (1, d)).astype(np.float32)).to(torch.bfloat16).cuda()
    b = torch.zeros(1, dtype=torch.float32, device="cuda")
    logit = torch.full((1, T), float("nan"), device="cuda")
    score = torch.full((1, T), float("nan"), device="cuda")
    px.xmix_probe_score(h, rt, w, b, [0], px.XMIX_PROBE_TOKEN, logit, score)
    before = (host_mask(rt), rt.app_count.cpu().numpy(), rt.app_tokens.cpu().numpy())
    thr = 0.25
    px.xmix_route_gate(rt, 1, logit[0].contiguous(),
                       torch.tensor([thr], dtype=torch.float32, device="cuda"), signal_bit=0)
    off = make_offsets(rng, 1, E)
    lg, lg_host = make_logits(rng, T, E, "bf16")
    px.xmix_router_write(lg, rt, [1], torch.from_numpy(off).cuda())
    sig = logit[0].cpu().numpy()
    tm2, _, _ = oracle.route_gate(*before, 1, sig, thr, signal_bit=0)
    ref = oracle.router_write(lg_host, tm2, [1], off)
    assert np.array_equal(host_bits(lg), ref)
    passed = sig >= thr
    assert 0 < passed.sum() < T
    assert np.array_equal(host_bits(lg)[~passed], lg_host[~passed])


def test_router_write_graph_replay_with_new_offsets(px):
    """The offsets live in device memory: one captured write serves new
    offsets without recapture (replayed with eager work and synchronisations
    between the replays, each checked)."""
    rng = np.random.default_rng(8)
    T, E = 512, 8
    sub = rng.integers(0, 8, T).astype(np.uint32)
    rt = gpu_route(px, np.arange(T, dtype=np.int32), T, sub, 3)
    lg0, lg_host = make_logits(rng, T, E, "bf16")
    lg = lg0.clone()
    off_d = torch.from_numpy(make_offsets(rng, 3, E)).cuda()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        px.xmix_router_write(lg, rt, [0, 1, 2], off_d)
    tm = host_mask(rt)
    for rep in range(3):
        off = make_offsets(rng, 3, E)
        off_d.copy_(torch.from_numpy(off))
        lg.copy_(lg0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        ref = oracle.router_write(lg_host, tm, [0, 1, 2], off)
        assert np.array_equal(host_bits(lg), ref), f"replay {rep}"
