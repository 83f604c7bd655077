"""GPU (HIP, gfx950) vs CPU oracle, stage by stage, at sizes the oracle
finishes in seconds.  Every call goes through the C ABI via the binding.

Sizes span several tiles and a ragged tail: T not a multiple of 64 or of
the 128-token encode tile, m several 256-latent tiles, padding tokens."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import (bf16_f64, check_delta, check_probe, check_residual, check_steer,
                    check_topk, torch_bits)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def px():
    import paper_2607_22595_amd as px
    return px


def dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def dev_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a).astype(np.uint32).view(np.int32)
                            if np.asarray(a).dtype == np.uint32 else
                            np.ascontiguousarray(a, np.int32)).cuda()


def gpu_route(px, req, T_valid, sub, n_apps):
    rt = px.Route(len(req), n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_build(dev_i32(req), torch.tensor([T_valid], dtype=torch.int32, device="cuda"),
                        dev_i32(np.asarray(sub, np.uint32)), rt, err)
    torch.cuda.synchronize()
    return rt, err


# -------------------------------------------------------------------- route

@pytest.mark.parametrize("seed", range(10))
def test_route_bit_exact(px, seed):
    rng = np.random.default_rng(100 + seed)
    T_max = int(rng.choice([1, 17, 64, 65, 1000, 1024, 1500, 8192]))
    R = int(rng.integers(1, 600))
    n_apps = int(rng.integers(1, 33))
    req = rng.integers(-2, R + 2, T_max).astype(np.int32)
    sub = rng.integers(0, 2 ** 32, R, dtype=np.uint64).astype(np.uint32)
    T_valid = int(rng.choice([T_max, max(T_max - 7, 0), -1, T_max + 3]))
    rt, err = gpu_route(px, req, T_valid, sub, n_apps)
    tm, cnt, lists, e = oracle.route(req, T_valid, sub, n_apps)
    assert np.array_equal(rt.tok_mask.cpu().numpy().view(np.uint32), tm)
    assert np.array_equal(rt.app_count.cpu().numpy(), cnt)
    assert np.array_equal(rt.app_tokens.cpu().numpy(), lists)
    assert int(err.item()) == e


@pytest.mark.parametrize("fill", [0, 0xFFFFFFFF])
def test_route_all_zero_and_all_one_masks(px, fill):
    T = 300
    req = np.arange(T, dtype=np.int32) % 77
    sub = np.full(77, fill, np.uint32)
    rt, err = gpu_route(px, req, T, sub, 32)
    tm, cnt, lists, e = oracle.route(req, T, sub, 32)
    assert np.array_equal(rt.app_tokens.cpu().numpy(), lists) and int(err.item()) == e == 0
    assert np.array_equal(rt.app_count.cpu().numpy(), cnt)


# ----------------------------------------------------------------- steering

def _steer_case(px, wl, layer=0, alpha=None):
    L = wl.layers[layer]
    tm, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    a = wl.alpha if alpha is None else alpha
    bits = [s.bit for s in L.steer]
    v = np.stack([s.v for s in L.steer])
    if wl.dtype == "bf16":
        h = dev_bits(L.h)
        vd = dev_bits(v)
    else:
        h = torch.from_numpy(L.h.copy()).cuda()
        vd = torch.from_numpy(v).cuda()
    px.xmix_steer_apply(h, rt, dev_i32(wl.req), vd, bits, torch.from_numpy(a).cuda())
    torch.cuda.synchronize()
    ref = oracle.steer(L.h, tm, wl.req, v, bits, a)
    rows = (tm & np.uint32(sum(1 << b for b in bits))) != 0
    got = torch_bits(h) if wl.dtype == "bf16" else h.cpu().numpy()
    return check_steer(got, ref, L.h, rows, wl.dtype == "bf16")


def test_steer_toy_fp32(px):
    _steer_case(px, synth.make("c1"))


def test_steer_decode_8b_shape(px):
    wl = synth.make("c2", n_layers=2)
    for layer in range(2):
        _steer_case(px, wl, layer)


def test_steer_alpha_zero_is_identity(px):
    wl = synth.make("c2", d=512, T=100, n_layers=1)
    L = wl.layers[0]
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    h = dev_bits(L.h)
    px.xmix_steer_apply(h, rt, dev_i32(wl.req), dev_bits(np.stack([s.v for s in L.steer])),
                        [s.bit for s in L.steer], torch.zeros_like(torch.from_numpy(wl.alpha)).cuda())
    assert np.array_equal(bf16_f64(torch_bits(h)), bf16_f64(L.h))


def test_steer_70b_shape_16_vectors(px):
    wl = synth.make("c5", m=256, k=8)   # steering and probes at full size
    _steer_case(px, wl)


def test_steer_padding_and_ragged(px):
    wl = synth.make("c2", d=264 - 8, T=77, n_layers=1)
    wl.req[70:] = -1
    wl.T_valid = 70
    _steer_case(px, wl)


# ------------------------------------------------------------------- probes

def _probe_case(px, wl, layer=0):
    L = wl.layers[layer]
    tm, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    h = dev_bits(L.h) if wl.dtype == "bf16" else torch.from_numpy(L.h).cuda()
    hv = bf16_f64(L.h) if wl.dtype == "bf16" else L.h.astype(np.float64)
    for mode_name, mode in (("token", px.XMIX_PROBE_TOKEN), ("mean", px.XMIX_PROBE_MEAN),
                            ("last", px.XMIX_PROBE_LAST)):
        ps = [p for p in L.probes if p.mode == mode_name]
        if not ps:
            continue
        w = np.stack([p.w for p in ps])
        b = np.array([p.b for p in ps], np.float32)
        bits = [p.bit for p in ps]
        n_out = wl.T_max if mode == px.XMIX_PROBE_TOKEN else wl.R_max
        lo = torch.full((len(ps), n_out), float("nan"), device="cuda")
        so = torch.full((len(ps), n_out), float("nan"), device="cuda")
        nb = px.probe_workspace(wl.T_max, len(ps), mode)
        ws = torch.empty(max(nb, 1), dtype=torch.uint8, device="cuda")
        wd = dev_bits(w) if wl.dtype == "bf16" else torch.from_numpy(w).cuda()
        cu = None if wl.cu_seqlens is None else dev_i32(wl.cu_seqlens)
        px.xmix_probe_score(h, rt, wd, torch.from_numpy(b).cuda(), bits, mode, lo, so,
                            cu_seqlens=cu, ws=ws)
        torch.cuda.synchronize()
        wv = bf16_f64(w) if wl.dtype == "bf16" else w.astype(np.float64)
        absdot = np.abs(wv) @ np.abs(hv).T        # [n_probe, T]
        if mode == px.XMIX_PROBE_TOKEN:
            lr, sr = oracle.probe_token(L.h, tm, w, b, bits)
            floor = absdot
        elif mode == px.XMIX_PROBE_LAST:
            lr, sr = oracle.probe_last(L.h, tm, w, b, bits, wl.cu_seqlens)
            cu = wl.cu_seqlens
            floor = np.stack([[absdot[p, cu[r + 1] - 1] if cu[r + 1] > cu[r] else 0.0
                               for r in range(wl.R_max)] for p in range(len(ps))])
        else:
            lr, sr = oracle.probe_mean(L.h, tm, w, b, bits, wl.cu_seqlens)
            cu = wl.cu_seqlens
            floor = np.stack([[absdot[p, cu[r]:cu[r + 1]].mean() if cu[r + 1] > cu[r] else 0.0
                               for r in range(wl.R_max)] for p in range(len(ps))])
        written = ~np.isnan(lr)
        lg, sg = lo.cpu().numpy(), so.cpu().numpy()
        assert np.all(np.isnan(lg[~written])), "unsubscribed outputs were written"
        check_probe(lg, sg, lr, sr, written, floor)


def test_probe_toy_fp32(px):
    _probe_case(px, synth.make("c1"))


def test_probe_decode_8b_shape(px):
    _probe_case(px, synth.make("c2", n_layers=1))


def test_probe_prefill_token_and_pooled_small(px):
    _probe_case(px, synth.make("c4", d=512, T=2000, R=5, len_lo=100, len_hi=700, m=256, k=8))


def test_probe_last_token_with_empty_and_unsubscribed_spans(px):
    """Last-token reads: one output per request from the last token of its
    span; an empty span and an unsubscribed request are not written."""
    wl = synth.make("c4", d=512, T=1200, R=6, len_lo=100, len_hi=400, m=256, k=8, n_last=3)
    cu = wl.cu_seqlens.copy()
    cu[3] = cu[2]                       # request 2 gets an empty span ...
    wl.cu_seqlens = cu
    wl.req[cu[3]:cu[4]] = 3             # ... and request 3 takes its tokens
    wl.sub[4] &= ~np.uint32(1 << 10)    # request 4 drops one last-token probe
    _probe_case(px, wl)


def test_probe_70b_shape(px):
    _probe_case(px, synth.make("c5", m=256, k=8))


def _pooled_case(px, wl, narrow=None):
    """Mean-pooled probes of wl's layer 0 against the oracle on a route that
    `narrow(rt, tm, cnt, lists)` may narrow first (GPU) and returns the
    oracle's narrowed mask for.  The workspace starts as NaN bit patterns, so
    a span sum that read a token the pass skipped is NaN."""
    L = wl.layers[0]
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    if narrow is not None:
        tm = narrow(rt, tm, cnt, lists)
    ps = [p for p in L.probes if p.mode == "mean"]
    w = np.stack([p.w for p in ps])
    b = np.array([p.b for p in ps], np.float32)
    bits = [p.bit for p in ps]
    lo = torch.full((len(ps), wl.R_max), float("nan"), device="cuda")
    so = torch.full((len(ps), wl.R_max), float("nan"), device="cuda")
    ws = torch.full((px.probe_workspace(wl.T_max, len(ps), px.XMIX_PROBE_MEAN),), 0xFF,
                    dtype=torch.uint8, device="cuda")
    px.xmix_probe_score(dev_bits(L.h), rt, dev_bits(w), torch.from_numpy(b).cuda(), bits,
                        px.XMIX_PROBE_MEAN, lo, so, cu_seqlens=dev_i32(wl.cu_seqlens), ws=ws)
    torch.cuda.synchronize()
    lr, sr = oracle.probe_mean(L.h, tm, w, b, bits, wl.cu_seqlens)
    cu = wl.cu_seqlens
    absdot = np.abs(bf16_f64(w)) @ np.abs(bf16_f64(L.h)).T
    floor = np.stack([[absdot[q, cu[r]:cu[r + 1]].mean() if cu[r + 1] > cu[r] else 0.0
                       for r in range(wl.R_max)] for q in range(len(ps))])
    written = ~np.isnan(lr)
    lg, sg = lo.cpu().numpy(), so.cpu().numpy()
    assert np.array_equal(np.isnan(lg), ~written), "written set differs from the oracle's"
    check_probe(lg, sg, lr, sr, written, floor)
    return written


def _small_prefill():
    return synth.make("c4", d=512, T=2000, R=5, len_lo=100, len_hi=700, m=256, k=8)


def test_probe_mean_span_past_t_valid(px):
    """T_valid ends inside the last span: the request is pooled (its first
    token is live) over its whole span, tokens past T_valid included."""
    wl = _small_prefill()
    cu = wl.cu_seqlens
    wl.T_valid = int(cu[-2] + (cu[-1] - cu[-2]) // 3)
    written = _pooled_case(px, wl)
    assert written[:, -1].all()


def test_probe_mean_with_padding_inside_a_span(px):
    """Padding slots (request -1, mask 0) inside a span still count."""
    wl = _small_prefill()
    cu = wl.cu_seqlens
    wl.req[cu[1] + 5:cu[1] + 40] = -1
    wl.req[cu[3] - 3:cu[3]] = -1
    written = _pooled_case(px, wl)
    assert written[:, 1].all() and written[:, 2].all()


def test_probe_mean_after_a_trigger_clears_the_bit_mid_span(px):
    """A token-driven filter clears a pooled probe's bit on some tokens of a
    span: a request whose first token keeps the bit is pooled over its whole
    span; one whose first token loses it is not written."""
    wl = _small_prefill()
    cu, T = wl.cu_seqlens, wl.T_max
    bit = [p.bit for p in wl.layers[0].probes if p.mode == "mean"][1]
    V = 1000
    rng = np.random.default_rng(7)
    ids = rng.integers(0, V, T).astype(np.int32)
    trig = np.arange(0, V, 2)                      # even ids pass
    vocab = np.zeros((V + 31) // 32, np.uint32)
    np.bitwise_or.at(vocab, trig >> 5, (np.uint32(1) << (trig & 31).astype(np.uint32)))
    ids[cu[0]] = 4                                  # request 0: first token passes
    ids[cu[1]] = 3                                  # request 1: first token fails
    ids[cu[2]] = 10
    ids[cu[2] + 1:cu[3]] = 11                       # request 2: only its first token passes

    def narrow(rt, tm, cnt, lists):
        px.xmix_route_trigger(rt, bit, dev_i32(ids), dev_i32(vocab), V)
        return oracle.route_trigger(tm, cnt, lists, bit, ids, vocab, V)[0]

    written = _pooled_case(px, wl, narrow)
    q = [p.bit for p in wl.layers[0].probes if p.mode == "mean"].index(bit)
    assert written[q, 0] and not written[q, 1] and written[q, 2]


# ------------------------------------------------- probes + steering, fused

def _steer_probe_case(px, wl, layer=0):
    """One fused pass against the two separate calls (bit-identical rows and
    probe outputs) and against the oracle (the probes see the row as read)."""
    L = wl.layers[layer]
    tm, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    bf = wl.dtype == "bf16"
    put = (lambda a: dev_bits(a)) if bf else (lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda())
    ps = [p for p in L.probes if p.mode == "token"]
    sbits, pbits = [s.bit for s in L.steer], [p.bit for p in ps]
    v, w = np.stack([s.v for s in L.steer]), np.stack([p.w for p in ps])
    b = np.array([p.b for p in ps], np.float32)
    vd, wd, bd = put(v), put(w), torch.from_numpy(b).cuda()
    alpha, req = torch.from_numpy(wl.alpha).cuda(), dev_i32(wl.req)
    nan = lambda: torch.full((len(ps), wl.T_max), float("nan"), device="cuda")
    # separate calls: probes first (they read the activation as produced)
    h1, l1, s1 = put(L.h), nan(), nan()
    px.xmix_probe_score(h1, rt, wd, bd, pbits, px.XMIX_PROBE_TOKEN, l1, s1)
    px.xmix_steer_apply(h1, rt, req, vd, sbits, alpha)
    h2, l2, s2 = put(L.h), nan(), nan()
    px.xmix_steer_probe(h2, rt, req, vd, sbits, alpha, wd, bd, pbits, l2, s2)
    torch.cuda.synchronize()
    g1 = torch_bits(h1) if bf else h1.cpu().numpy()
    g2 = torch_bits(h2) if bf else h2.cpu().numpy()
    assert np.array_equal(g1.view(np.uint8), g2.view(np.uint8))
    for a, c in ((l1, l2), (s1, s2)):
        a, c = a.cpu().numpy(), c.cpu().numpy()
        assert np.array_equal(np.isnan(a), np.isnan(c))
        assert np.array_equal(a[~np.isnan(a)].view(np.uint32), c[~np.isnan(c)].view(np.uint32))
    # against the oracle
    ref = oracle.steer(L.h, tm, wl.req, v, sbits, wl.alpha)
    rows = (tm & np.uint32(sum(1 << q for q in sbits))) != 0
    check_steer(g2, ref, L.h, rows, bf)
    lr, sr = oracle.probe_token(L.h, tm, w, b, pbits)
    hv = bf16_f64(L.h) if bf else L.h.astype(np.float64)
    wv = bf16_f64(w) if bf else w.astype(np.float64)
    written = ~np.isnan(lr)
    lg, sg = l2.cpu().numpy(), s2.cpu().numpy()
    assert np.all(np.isnan(lg[~written])), "unsubscribed outputs were written"
    check_probe(lg, sg, lr, sr, written, np.abs(wv) @ np.abs(hv).T)


@pytest.mark.parametrize("d,T,t_valid,bad_ids", [
    (4096, 256, 256, False),    # the 8B-shaped decode layer
    (256, 300, 290, True),      # padding and bad request ids
    (256, 40, 45, False),       # T_valid above T_max (error bit 2)
    (256, 6, 6, False),         # fewer slots than apps: a route launch first
    (256, 1100, 1100, True)])   # over 1024 slots: a route launch first
def test_route_built_inside_the_steer_probe_pass(px, d, T, t_valid, bad_ids):
    """xmix_route_steer_probe leaves the route, the error word, the rows and
    the probe outputs exactly as xmix_route_build followed by
    xmix_steer_probe; the routing is also checked against the oracle."""
    wl = synth.make("c2", d=d, T=T, n_layers=1)
    L = wl.layers[0]
    rng = np.random.default_rng(T)
    req = wl.req.copy()
    if bad_ids:
        req[rng.choice(T, 7, replace=False)] = wl.sub.size + 3
        req[rng.choice(T, 5, replace=False)] = -1
    sub = wl.sub | np.uint32(1 << 30)   # a bit beyond n_apps is dropped
    ps = [p for p in L.probes if p.mode == "token"]
    sbits, pbits = [q.bit for q in L.steer], [q.bit for q in ps]
    vd = dev_bits(np.stack([q.v for q in L.steer]))
    wd = dev_bits(np.stack([q.w for q in ps]))
    bd = torch.tensor([q.b for q in ps], dtype=torch.float32, device="cuda")
    alpha = torch.from_numpy(wl.alpha).cuda()
    tv = torch.tensor([t_valid], dtype=torch.int32, device="cuda")
    reqd, subd = dev_i32(req), dev_i32(sub)
    outs = []
    for fused in (False, True):
        rt = px.Route(T, wl.n_apps)
        rt.tok_mask.fill_(-5)
        rt.app_count.fill_(-5)
        rt.app_tokens.fill_(-5)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        h = dev_bits(L.h)
        lo = torch.full((len(ps), T), float("nan"), device="cuda")
        so = torch.full((len(ps), T), float("nan"), device="cuda")
        if fused:
            px.xmix_route_steer_probe(reqd, tv, subd, rt, err, h, vd, sbits, alpha, wd, bd, pbits,
                                      lo, so)
        else:
            px.xmix_route_build(reqd, tv, subd, rt, err)
            px.xmix_steer_probe(h, rt, reqd, vd, sbits, alpha, wd, bd, pbits, lo, so)
        torch.cuda.synchronize()
        outs.append((rt.tok_mask.cpu().numpy().view(np.uint32), rt.app_count.cpu().numpy(),
                     rt.app_tokens.cpu().numpy(), int(err.item()), torch_bits(h),
                     lo.cpu().numpy().view(np.uint32), so.cpu().numpy().view(np.uint32)))
    for a, b in zip(*outs):
        assert np.array_equal(np.asarray(a), np.asarray(b))
    tm, cnt, lists, e = oracle.route(req, t_valid, sub, wl.n_apps)
    assert np.array_equal(outs[1][0], tm) and np.array_equal(outs[1][1], cnt)
    assert np.array_equal(outs[1][2], lists) and outs[1][3] == e


def test_steer_probe_fused_toy_fp32(px):
    _steer_probe_case(px, synth.make("c1"))


def test_steer_probe_fused_decode_8b_shape(px):
    wl = synth.make("c2", n_layers=2)
    for layer in range(2):
        _steer_probe_case(px, wl, layer)


def test_steer_probe_fused_padding_and_ragged(px):
    wl = synth.make("c2", d=264 - 8, T=77, n_layers=1)
    wl.req[70:] = -1
    wl.T_valid = 70
    _steer_probe_case(px, wl)


def test_steer_probe_fused_70b_shape(px):
    _steer_probe_case(px, synth.make("c5", m=256, k=8))


# --------------------------------------------------------------- SAE encode

def _encode(px, wl, sae, h_bits, fold=True):
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    h = dev_bits(h_bits)
    W = px.xmix_sae_pack_encoder(dev_bits(sae.W_enc))
    be, bd = dev_bits(sae.b_enc), dev_bits(sae.b_dec)
    c = None
    if fold:
        c = torch.empty(sae.m, dtype=torch.float32, device="cuda")
        px.xmix_sae_fold_bias(W, be, bd, c)
    idx = torch.full((wl.T_max, sae.k), -7, dtype=torch.int32, device="cuda")
    val = torch.zeros((wl.T_max, sae.k), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(px.sae_encode_workspace(wl.T_max, wl.d, sae.m, sae.k), dtype=torch.uint8,
                     device="cuda")
    px.xmix_sae_encode_topk(h, rt, sae.bit, W, be, bd, c, sae.k, idx, val, ws)
    torch.cuda.synchronize()
    return rt, idx.cpu().numpy(), torch_bits(val)


def _check_encode(wl, sae, h_bits, idx, val, tokens):
    idx_ref, _, _, pre = oracle.sae_encode(h_bits, tokens, sae.W_enc, sae.b_enc, sae.b_dec,
                                           sae.k, want_pre=True)
    swaps = 0
    for q, t in enumerate(tokens):
        swaps += check_topk(idx[t], val[t], idx_ref[q], pre[q], sae.k)
    return swaps


@pytest.mark.parametrize("d,m,k,T", [(256, 1024, 16, 64), (512, 2048, 64, 200), (768, 768, 1, 37),
                                     (256, 256, 64, 130)])
def test_encode_topk_small(px, d, m, k, T):
    wl = synth.make("c3", d=d, m=m, k=k, T=T)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    toks = lists[0, :cnt[0]]
    _check_encode(wl, sae, wl.layers[0].h, idx, val, toks)
    # unsubscribed rows are not written
    off = np.setdiff1d(np.arange(T), toks)
    assert np.all(idx[off] == -7)


def test_encode_without_folded_bias(px):
    wl = synth.make("c3", d=256, m=512, k=32, T=50)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h, fold=False)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, lists[0, :cnt[0]])


def test_encode_all_tokens_many_token_tiles(px):
    # every token subscribed, 3 token tiles with a ragged last tile
    wl = synth.make("c3", d=256, m=1024, k=8, T=300, n_sub=300)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, np.arange(300))


def test_encode_decode_kernel_blocked_tile_order(px):
    """Between 513 and 1024 token slots the decode kernel walks its tiles in
    XCD blocks of 8 token tiles x 4 latent tiles (more than 4 token tiles);
    900 slots with 777 subscribed leave a ragged last token tile."""
    wl = synth.make("c3", d=256, m=2048, k=16, T=900, n_sub=777)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    toks = lists[0, :cnt[0]]
    assert len(toks) == 777
    _check_encode(wl, sae, wl.layers[0].h, idx, val, toks)
    off = np.setdiff1d(np.arange(900), toks)
    assert np.all(idx[off] == -7)


@pytest.mark.parametrize("d,m,k,T,n_sub", [(256, 1024, 16, 1500, 1100), (512, 2048, 32, 2100, 2100),
                                           (256, 2560, 64, 1025, 700)])
def test_encode_prefill_gemm_path(px, d, m, k, T, n_sub):
    """From 1025 token slots the encode stages the token rows and runs the
    256 x 256-tile GEMM; ragged subscribed counts leave a partial last tile
    and padded token planes."""
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=n_sub)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    toks = lists[0, :cnt[0]]
    assert len(toks) == n_sub
    _check_encode(wl, sae, wl.layers[0].h, idx, val, toks)
    off = np.setdiff1d(np.arange(T), toks)
    assert np.all(idx[off] == -7)


def test_encode_prefill_gemm_no_subscribers(px):
    wl = synth.make("c3", d=256, m=512, k=8, T=1100, n_sub=0)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    assert np.all(idx == -7)


@pytest.mark.parametrize("T", [40, 1100])
def test_encode_exact_ties_take_lower_index(px, T):
    """Duplicated dictionary rows give bit-identical pre-activations; the
    lower latent index must win, across tiles and inside one tile (40 token
    slots run the decode kernel, 1100 the prefill GEMM)."""
    wl = synth.make("c3", d=256, m=1024, k=16, T=T)
    sae = wl.layers[0].saes[0]
    W = sae.W_enc.copy()
    b = sae.b_enc.copy()
    for src, dst in ((5, 900), (5, 6), (300, 301), (300, 1000), (77, 513)):
        W[dst] = W[src]
        b[dst] = b[src]
    sae.W_enc, sae.b_enc = W, b
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    toks = lists[0, :cnt[0]]
    _check_encode(wl, sae, wl.layers[0].h, idx, val, toks)
    for t in toks:
        s = set(idx[t].tolist())
        for lo_, hi_ in ((5, 900), (5, 6), (300, 301), (300, 1000), (77, 513)):
            if hi_ in s:
                assert lo_ in s, f"token {t}: {hi_} selected without its lower twin {lo_}"


@pytest.mark.parametrize("shift,T,n_sub", [(-60.0, 40, None), (-12.0, 40, None),
                                           (-60.0, 1100, 1100), (-12.0, 1100, 1000)])
def test_encode_negative_pre_activations(px, shift, T, n_sub):
    """b_enc moved down so that every pre-activation is negative (-60), or so
    that fewer than k are positive (-12): the k largest are still taken by
    value (ties to the lower latent) and the negative ones come out as 0."""
    # 40 token slots run the decode kernel; 1100 run the prefill GEMM
    kw = {} if n_sub is None else {"n_sub": n_sub}
    wl = synth.make("c3", d=256, m=1024, k=16, T=T, **kw)
    sae = wl.layers[0].saes[0]
    b = torch.from_numpy(bf16_f64(sae.b_enc) + shift).float().to(torch.bfloat16)
    sae.b_enc = b.view(torch.int16).numpy().view(np.uint16)
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    toks = lists[0, :cnt[0]]
    _check_encode(wl, sae, wl.layers[0].h, idx, val, toks)
    _, _, _, pre = oracle.sae_encode(wl.layers[0].h, toks, sae.W_enc, sae.b_enc, sae.b_dec,
                                     sae.k, want_pre=True)
    n_pos = (pre > 0).sum(axis=1)
    if shift == -60.0:
        assert n_pos.max() == 0 and np.all(val[toks] == 0)
    else:
        assert n_pos.min() < sae.k  # the k-th value is negative for some tokens


@pytest.mark.parametrize("T,n_apps,bit,t_valid,bad_ids,m", [
    (256, 1, 0, 256, False, 1024),    # the decode SAE step: one app
    (300, 3, 2, 290, True, 1024),     # the SAE on bit 2 of 3, padding and bad ids
    (40, 2, 0, 45, False, 1024),      # T_valid above T_max (error bit 2)
    (1000, 5, 1, 1000, True, 1024),   # up to the in-kernel limit
    (40, 3, 1, 40, False, 256),       # one workgroup, three apps: a route launch
    (1100, 2, 0, 1100, False, 1024)])  # over 1024 slots: a route launch
def test_route_built_inside_the_encode(px, T, n_apps, bit, t_valid, bad_ids, m):
    """xmix_route_sae_encode_candidates leaves the route, the error word and
    (after the merge) the top-k exactly as xmix_route_build followed by the
    candidates stage does; the routing is also checked against the oracle."""
    wl = synth.make("c3", d=256, m=m, k=16, T=T)
    sae = wl.layers[0].saes[0]
    rng = np.random.default_rng(T + n_apps)
    sub = (wl.sub & np.uint32(1)) << np.uint32(bit)
    for a in range(n_apps):
        if a != bit:
            sub |= (rng.random(wl.sub.size) < 0.4).astype(np.uint32) << np.uint32(a)
    sub |= np.uint32(1 << 31)     # a bit beyond n_apps is dropped
    req = wl.req.copy()
    if bad_ids:
        req[rng.choice(T, 7, replace=False)] = wl.sub.size + 3   # >= R_max
        req[rng.choice(T, 5, replace=False)] = -1
    h = dev_bits(wl.layers[0].h)
    W = px.xmix_sae_pack_encoder(dev_bits(sae.W_enc))
    be, bd = dev_bits(sae.b_enc), dev_bits(sae.b_dec)
    c = torch.empty(sae.m, dtype=torch.float32, device="cuda")
    px.xmix_sae_fold_bias(W, be, bd, c)
    tv = torch.tensor([t_valid], dtype=torch.int32, device="cuda")
    reqd, subd = dev_i32(req), dev_i32(sub)
    outs = []
    for fused in (False, True):
        rt = px.Route(T, n_apps)
        rt.tok_mask.fill_(-5)
        rt.app_count.fill_(-5)
        rt.app_tokens.fill_(-5)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        ws = torch.empty(px.sae_encode_workspace(T, wl.d, sae.m, sae.k), dtype=torch.uint8,
                         device="cuda")
        idx = torch.full((T, sae.k), -7, dtype=torch.int32, device="cuda")
        val = torch.zeros((T, sae.k), dtype=torch.bfloat16, device="cuda")
        if fused:
            px.xmix_route_sae_encode_candidates(reqd, tv, subd, rt, err, h, bit, W, be, bd, c,
                                                sae.k, ws)
        else:
            px.xmix_route_build(reqd, tv, subd, rt, err)
            px.xmix_sae_encode_candidates(h, rt, bit, W, be, bd, c, sae.k, ws)
        px.xmix_sae_merge_topk(h, rt, bit, W, c, sae.k, idx, val, ws)
        torch.cuda.synchronize()
        outs.append((rt.tok_mask.cpu().numpy().view(np.uint32), rt.app_count.cpu().numpy(),
                     rt.app_tokens.cpu().numpy(), int(err.item()), idx.cpu().numpy(),
                     torch_bits(val)))
    for a, b in zip(*outs):
        assert np.array_equal(np.asarray(a), np.asarray(b))
    tm, cnt, lists, e = oracle.route(req, t_valid, sub, n_apps)
    assert np.array_equal(outs[1][0], tm) and np.array_equal(outs[1][1], cnt)
    assert np.array_equal(outs[1][2], lists) and outs[1][3] == e
    assert cnt[bit] > 0


def test_encode_clustered_winners_in_one_tile(px):
    """All k winners planted in one 256-latent tile."""
    d, m, k = 256, 1024, 64
    wl = synth.make("c3", d=d, m=m, k=k, T=20, n_sub=20)
    sae = wl.layers[0].saes[0]
    hv = bf16_f64(wl.layers[0].h)
    W = sae.W_enc.copy()
    t0 = 3
    for r in range(k):
        row = hv[t0] * 3.0 * (1.0 - 0.004 * r) / d
        W[512 + r] = torch.from_numpy(row.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    sae.W_enc = W
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, np.arange(20))
    assert set(idx[t0].tolist()) == set(range(512, 512 + k))


def test_encode_no_subscribers_writes_nothing(px):
    wl = synth.make("c3", d=256, m=512, k=8, T=64, n_sub=0)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    assert np.all(idx == -7)


# ------------------------------------------------------------- clamp-decode

@pytest.mark.parametrize("d,m,k,T", [(256, 1024, 16, 64), (512, 768, 64, 90)])
def test_clamp_decode_stage_isolated(px, d, m, k, T):
    wl = synth.make("c5", d=d, T=T, m=m, k=k, p=0.5)
    L = wl.layers[0]
    for sae in L.saes[:3]:
        rt, idx, val = _encode(px, wl, sae, L.h)
        tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
        # make one clamp id hit a selected feature of the first subscribed token
        ids = sae.clamp_ids.copy()
        if cnt[sae.bit]:
            ids[0] = idx[lists[sae.bit, 0], 0]
        h = dev_bits(L.h)
        delta = torch.zeros((T, d), dtype=torch.float32, device="cuda")
        px.xmix_sae_clamp_decode(h, rt, sae.bit, torch.from_numpy(idx).cuda(),
                                 dev_bits(val), dev_bits(sae.W_dec), dev_i32(ids),
                                 torch.from_numpy(sae.clamp_vals).cuda(), delta)
        torch.cuda.synchronize()
        ref, dref = oracle.clamp_decode(L.h, tm, sae.bit, idx, val, sae.W_dec, ids,
                                        sae.clamp_vals, want_delta=True)
        rows = (tm >> np.uint32(sae.bit)) & 1 == 1
        got = torch_bits(h)
        assert np.array_equal(got[~rows], L.h[~rows])
        dg = delta.cpu().numpy()
        for t in np.nonzero(rows)[0]:
            check_delta(dg[t], dref[t])
            check_residual(got[t], ref[t], dref[t])


def test_clamp_to_current_value_leaves_h(px):
    wl = synth.make("c5", d=256, T=32, m=512, k=8, p=1.0)
    L = wl.layers[0]
    sae = L.saes[0]
    rt, idx, val = _encode(px, wl, sae, L.h)
    # clamp token 0's own top-4 features to the values it already has: delta = 0
    cids = idx[0, :4].copy()
    cvals = bf16_f64(val[0, :4]).astype(np.float32)
    h = dev_bits(L.h)
    only_t0 = np.array([0] + [-1] * (wl.T_max - 1), np.int32)
    rt1, _ = gpu_route(px, only_t0, wl.T_max, wl.sub, wl.n_apps)
    px.xmix_sae_clamp_decode(h, rt1, sae.bit, torch.from_numpy(idx).cuda(), dev_bits(val),
                             dev_bits(sae.W_dec), dev_i32(cids), torch.from_numpy(cvals).cuda())
    torch.cuda.synchronize()
    assert np.array_equal(bf16_f64(torch_bits(h)), bf16_f64(L.h))


# ---------------------------------------------------------------- readback

@pytest.mark.parametrize("k", [16, 5])
def test_readback_ring_bit_exact_with_wraparound(px, k):
    """Odd k: rows of 16 + 6 k bytes, every other one 2 bytes past a 4-byte
    boundary."""
    wl = synth.make("c3", d=256, m=512, k=k, T=100, ring_capacity=64)
    sae = wl.layers[0].saes[0]
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    ring = px.Ring(64, 16 + k * 6)
    tm = rt.tok_mask.cpu().numpy().view(np.uint32)
    slots = np.zeros((64, 16 + k * 6), np.uint8)
    head = 0
    idx_d, val_d = torch.from_numpy(idx).cuda(), dev_bits(val)
    for step in range(3):   # 3 x 50 rows into 64 slots: wraps and overwrites
        px.xmix_readback_compact([idx_d, val_d], rt, sae.bit, dev_i32(wl.req), 7, sae.bit, ring)
        torch.cuda.synchronize()
        slots, head = oracle.compact([idx.view(np.uint8).reshape(wl.T_max, -1),
                                      val.view(np.uint8).reshape(wl.T_max, -1)],
                                     tm, sae.bit, wl.req, 7, sae.bit, slots, head)
        assert int(ring.head[0].item()) == head
        assert int(ring.head[1].item()) == 0
        assert np.array_equal(ring.slots.cpu().numpy(), slots)


def test_readback_more_rows_than_capacity(px):
    T = 300
    req = np.arange(T, dtype=np.int32)
    sub = np.ones(T, np.uint32)
    rt, _ = gpu_route(px, req, T, sub, 1)
    rows = np.arange(T * 8, dtype=np.int32).reshape(T, 8)
    ring = px.Ring(100, 16 + 32)
    px.xmix_readback_compact([torch.from_numpy(rows).cuda()], rt, 0, dev_i32(req), 1, 0, ring)
    torch.cuda.synchronize()
    slots, head = oracle.compact([rows.view(np.uint8).reshape(T, -1)], np.ones(T, np.uint32), 0,
                                 req, 1, 0, np.zeros((100, 48), np.uint8), 0)
    assert head == int(ring.head[0].item()) == 300
    assert np.array_equal(ring.slots.cpu().numpy(), slots)


@pytest.mark.parametrize("T,n_sub,cap,k", [(100, 50, 64, 16), (1500, 1100, 500, 8),
                                           (100, 50, 64, 7)])
def test_encode_with_fused_readback_bit_exact(px, T, n_sub, cap, k):
    """The merge writes the ring rows itself: same rows and head as the
    compaction of the encode's own outputs (3 calls: wrap-around and, in the
    second case, more rows per call than slots, on the prefill GEMM path)."""
    wl = synth.make("c3", d=256, m=1024, k=k, T=T, n_sub=n_sub, ring_capacity=cap)
    sae = wl.layers[0].saes[0]
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    h = dev_bits(wl.layers[0].h)
    W = px.xmix_sae_pack_encoder(dev_bits(sae.W_enc))
    be, bd = dev_bits(sae.b_enc), dev_bits(sae.b_dec)
    c = torch.empty(sae.m, dtype=torch.float32, device="cuda")
    px.xmix_sae_fold_bias(W, be, bd, c)
    idx_d = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
    val_d = torch.zeros((T, k), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(px.sae_encode_workspace(T, wl.d, sae.m, k), dtype=torch.uint8, device="cuda")
    row = 16 + 6 * k
    ring = px.Ring(cap, row)
    tm = rt.tok_mask.cpu().numpy().view(np.uint32)
    slots = np.zeros((cap, row), np.uint8)
    head = 0
    for step in range(3):
        px.xmix_sae_encode_topk_ring(h, rt, sae.bit, W, be, bd, c, k, idx_d, val_d, ws,
                                     dev_i32(wl.req), 5, sae.bit, ring)
        torch.cuda.synchronize()
        idx, val = idx_d.cpu().numpy(), torch_bits(val_d)
        slots, head = oracle.compact([idx.view(np.uint8).reshape(T, -1),
                                      val.view(np.uint8).reshape(T, -1)],
                                     tm, sae.bit, wl.req, 5, sae.bit, slots, head)
        assert int(ring.head[0].item()) == head == (step + 1) * n_sub
        assert int(ring.head[1].item()) == 0
        assert np.array_equal(ring.slots.cpu().numpy(), slots)
    toks = np.flatnonzero(tm & 1)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, toks[:40])


def test_encode_recompute_path_when_winners_crowd_one_slice(px):
    """50 of a token's top-64 planted in one 256-latent slice: more than the
    slice may emit, so the merge's certificate fails for that token and the
    repair recomputes that slice; the result must still match."""
    d, m, k = 256, 16384, 64
    wl = synth.make("c3", d=d, m=m, k=k, T=8, n_sub=8)
    sae = wl.layers[0].saes[0]
    hv = bf16_f64(wl.layers[0].h)
    W = sae.W_enc.copy()
    t0 = 5
    for r in range(50):
        row = hv[t0] * 3.0 * (1.0 - 0.005 * r) / d
        W[4096 + r] = torch.from_numpy(row.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    sae.W_enc = W
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, np.arange(8))
    assert set(range(4096, 4096 + 50)) <= set(idx[t0].tolist())


def to_bf16_bits(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).view(torch.int16) \
        .numpy().view(np.uint16)


@pytest.mark.parametrize("n_tied,T", [(10, 6), (20, 6), (64, 6), (10, 1100), (64, 1100)])
def test_encode_repair_of_tied_slices(px, n_tied, T):
    """n_tied slices whose 256 pre-activations are all exactly 40 (zero
    dictionary rows, bias 40), far above every other latent.  No threshold
    splits a tie, so these slices emit nothing and fail the certificate.
    The merge redoes slices in the order of their bounds: the first tied
    slice gives the k winners, and every other tied slice, bounded by the
    same value at higher latents, cannot beat them (64: nothing is emitted
    at all, the pool starts empty).  The k lowest latents of the tie win.
    With 1100 token slots the prefill GEMM runs, whose threshold search on
    a tied slice uses every refinement round and then gives up."""
    d, m, k = 256, 16384, 64
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T)
    sae = wl.layers[0].saes[0]
    W, b = sae.W_enc.copy(), sae.b_enc.copy()
    slices = np.arange(64) if n_tied == 64 else 1 + 3 * np.arange(n_tied)
    for s in slices:
        W[256 * s:256 * (s + 1)] = 0
        b[256 * s:256 * (s + 1)] = 0x4220  # 40.0
    sae.W_enc, sae.b_enc = W, b
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, np.arange(T))
    first = 256 * int(slices[0])
    for t in range(T):
        assert sorted(idx[t].tolist()) == list(range(first, first + k))
        assert np.all(bf16_f64(val[t]) == 40.0)


@pytest.mark.parametrize("T", [6, 1100])
def test_encode_repair_takes_the_highest_bound_first(px, T):
    """Ten tied slices at different levels (zero rows; the i-th tied slice
    has bias 40 + 2i), so the highest tie sits in the last of them: the
    merge must redo that slice first and stop there.  Its k lowest latents
    win with value 58."""
    d, m, k = 256, 16384, 64
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T)
    sae = wl.layers[0].saes[0]
    W, b = sae.W_enc.copy(), sae.b_enc.copy()
    slices = 1 + 3 * np.arange(10)
    for i, s in enumerate(slices):
        W[256 * s:256 * (s + 1)] = 0
        b[256 * s:256 * (s + 1)] = to_bf16_bits(np.full(256, 40.0 + 2 * i))
    sae.W_enc, sae.b_enc = W, b
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, np.arange(T))
    first = 256 * int(slices[-1])
    for t in range(T):
        assert sorted(idx[t].tolist()) == list(range(first, first + k))
        assert np.all(bf16_f64(val[t]) == 58.0)


@pytest.mark.parametrize("T", [6, 1100])
def test_encode_repair_winners_over_two_tied_slices(px, T):
    """Three slices each hold 32 latents tied at 40 (zero rows, bias 40) far
    above the rest, with k = 64: the repair needs the first two slices (32
    winners each) and must not take the third's, which lose on the latent
    index."""
    d, m, k = 256, 16384, 64
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T)
    sae = wl.layers[0].saes[0]
    W, b = sae.W_enc.copy(), sae.b_enc.copy()
    for s in (2, 5, 9):
        W[256 * s:256 * s + 32] = 0
        b[256 * s:256 * s + 32] = 0x4220  # 40.0
    sae.W_enc, sae.b_enc = W, b
    rt, idx, val = _encode(px, wl, sae, wl.layers[0].h)
    _check_encode(wl, sae, wl.layers[0].h, idx, val, np.arange(T))
    want = list(range(512, 544)) + list(range(1280, 1312))
    for t in range(T):
        assert sorted(idx[t].tolist()) == want
        assert np.all(bf16_f64(val[t]) == 40.0)


@pytest.mark.parametrize("T", [64, 1100])
def test_encode_with_strong_latents_per_token(px, T):
    """Every token's row is moved along three dictionary rows so that those
    latents stand far above its others (as clamping features high does).
    64 token slots run the decode kernel, whose first threshold guess leaves
    such values out of the tile statistics; 1100 run the prefill GEMM, which
    keeps the plain statistics and leaves failures to the merge's repair.
    The top-k must match the oracle either way."""
    d, m, k = 256, 4096, 32
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T)
    sae = wl.layers[0].saes[0]
    Wf = bf16_f64(sae.W_enc)
    h = bf16_f64(wl.layers[0].h)
    picks = synth.randint("test/strong_latents", 3 * T, 0, m - 1).reshape(T, 3)
    for t in range(T):
        for j in picks[t]:
            h[t] += 60.0 * Wf[j] / np.dot(Wf[j], Wf[j])
    hb = to_bf16_bits(h)
    rt, idx, val = _encode(px, wl, sae, hb)
    _check_encode(wl, sae, hb, idx, val, np.arange(T))
    for t in range(T):
        assert set(picks[t].tolist()) <= set(idx[t].tolist())


@pytest.mark.parametrize("T", [64, 1100])
def test_encode_pool_overflow_with_exact_ties(px, T):
    """Every 256-latent slice holds 8 identical rows (one direction the
    tokens share, one bias), so each slice emits 8 candidates of exactly the
    same value far above the rest: 4096 tied candidates per token, twice the
    merge's pool.  No refill floor on the value alone can cut them; the
    floor on (value, latent) does, and the k lowest tied latents (slices 0-3)
    win.  64 token slots run the decode kernel, 1100 the prefill GEMM."""
    d, m, k = 256, 131072, 32
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T, n_outliers=0)
    sae = wl.layers[0].saes[0]
    Wf = bf16_f64(sae.W_enc).reshape(m, d)
    b = sae.b_enc.copy()
    u = bf16_f64(synth.normal_bf16("test/overflow_ties/u", (d,), 1.0))
    u /= np.linalg.norm(u)
    tied = (np.arange(m) % 256) < 8
    Wf[tied] = (10.0 / np.sqrt(d)) * u[None, :]
    b[tied] = 0
    sae.W_enc, sae.b_enc = to_bf16_bits(Wf), b
    h = bf16_f64(wl.layers[0].h) + 3.0 * np.sqrt(d) * u[None, :]
    hb = to_bf16_bits(h)
    rt, idx, val = _encode(px, wl, sae, hb)
    _check_encode(wl, sae, hb, idx, val, np.arange(T))
    want = [256 * s + j for s in range(4) for j in range(8)]
    for t in range(T):
        assert sorted(idx[t].tolist()) == want
        assert len(set(val[t].tolist())) == 1


@pytest.mark.parametrize("T", [64, 1100])
def test_encode_candidate_pool_overflow(px, T):
    """Every 256-latent slice holds a cluster of 7 latents about 4 stdev
    above its others for every token (rows along one direction the tokens
    share), so each slice's first threshold guess keeps about 7 candidates:
    with m=131072 (512 slices) a token's candidates far exceed the merge's
    2048-entry pool.  The merge refills its pool above the k-th best of the
    first 2048 (the candidate counts read from the workspace show the
    overflow), and the top-k must still match the oracle on every token.
    64 token slots run the decode kernel, 1100 the prefill GEMM."""
    d, m, k = 256, 131072, 32
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T, n_outliers=0)
    sae = wl.layers[0].saes[0]
    Wf = bf16_f64(sae.W_enc).reshape(m, d)
    u = bf16_f64(synth.normal_bf16("test/overflow/u", (d,), 1.0))
    u /= np.linalg.norm(u)
    lat = np.arange(m)
    cl = (lat % 256) < 7
    # other latents: pre ~ N(0, 5) with the shift below; cluster: 9 to 9.9
    gamma = (4.5 + 0.45 * synth.uniform01("test/overflow/scale", m)) / np.sqrt(d)
    Wf[cl] = gamma[cl][:, None] * u[None, :]
    sae.W_enc = to_bf16_bits(Wf)
    h = bf16_f64(wl.layers[0].h) + 2.0 * np.sqrt(d) * u[None, :]
    hb = to_bf16_bits(h)
    rt, _ = gpu_route(px, wl.req, wl.T_valid, wl.sub, wl.n_apps)
    hd = dev_bits(hb)
    W = px.xmix_sae_pack_encoder(dev_bits(sae.W_enc))
    be, bd = dev_bits(sae.b_enc), dev_bits(sae.b_dec)
    c = torch.empty(m, dtype=torch.float32, device="cuda")
    px.xmix_sae_fold_bias(W, be, bd, c)
    idx = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
    val = torch.zeros((T, k), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(px.sae_encode_workspace(T, d, m, k), dtype=torch.uint8, device="cuda")
    px.xmix_sae_encode_candidates(hd, rt, sae.bit, W, be, bd, c, k, ws)
    torch.cuda.synchronize()
    # workspace (white box): folded bias (m fp32, rounded up to 256 bytes),
    # candidate pairs [T][n_mt][cap] (8 bytes each), counts [T][n_mt] int32
    n_mt, cap = m // 256, 8
    fold = (m * 4 + 255) // 256 * 256
    cnt_off = fold + T * n_mt * cap * 8
    counts = ws[cnt_off:cnt_off + T * n_mt * 4].cpu().numpy().view(np.int32).reshape(T, n_mt)
    assert counts.max() <= cap and counts.sum(axis=1).min() > 2048
    px.xmix_sae_merge_topk(hd, rt, sae.bit, W, c, k, idx, val, ws)
    torch.cuda.synchronize()
    _check_encode(wl, sae, hb, idx.cpu().numpy(), torch_bits(val), np.arange(T))


@pytest.mark.parametrize("T,kind", [(64, "pareto"), (1100, "pareto"), (64, "lognormal")])
def test_encode_heavy_tailed_pre_activations(px, T, kind):
    """Dictionary rows scaled by Pareto(1.5) factors (capped at 200): a
    token's pre-activations over the latents are a scale mixture of normals
    with a power-law tail, so the first threshold guess from a slice's mean
    and stdev misjudges it (slices with a large factor overshoot the window
    and refine, the others keep few candidates).  The top-k must still match
    the oracle on every token; 64 token slots run the decode kernel, 1100 the
    prefill GEMM.  The log-normal case (row norms exp(1.5 N(0, 1))) stands
    for dictionaries whose rows differ in norm by orders of magnitude."""
    d, m, k = 256, 16384, 32
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=T, n_outliers=0)
    sae = wl.layers[0].saes[0]
    u = synth.uniform01("test/heavy/scale", m)
    if kind == "pareto":
        f = np.minimum((1.0 - u) ** (-1.0 / 1.5), 200.0)
    else:
        f = np.exp(1.5 * bf16_f64(synth.normal_bf16("test/heavy/lognormal", (m,), 1.0)))
    sae.W_enc = to_bf16_bits(bf16_f64(sae.W_enc).reshape(m, d) * f[:, None])
    h = wl.layers[0].h
    # the tail is there: excess kurtosis of one token's pre-activations
    _, _, _, pre = oracle.sae_encode(h, np.array([0]), sae.W_enc, sae.b_enc, sae.b_dec, k,
                                     want_pre=True)
    z = (pre[0] - pre[0].mean()) / pre[0].std()
    assert np.mean(z ** 4) > (10.0 if kind == "pareto" else 6.0)
    rt, idx, val = _encode(px, wl, sae, h)
    _check_encode(wl, sae, h, idx, val, np.arange(T))
