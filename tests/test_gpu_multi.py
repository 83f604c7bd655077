"""The batched SAE calls of one hook against one call per app.

xmix_sae_encode_topk_multi (and its routed form) must give every app the
same indices, values and ring rows, bit for bit, as one xmix_sae_encode_topk
or xmix_sae_encode_topk_ring call per app; xmix_sae_clamp_decode_multi must
leave h (and each delta) exactly as one xmix_sae_clamp_decode call per app
in the same order.  One app of each batch is also checked against the
oracle, so the comparison is not between two wrong answers."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_topk, torch_bits

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def px():
    import paper_2607_22595_amd as px
    return px


def dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def dev_i32(a):
    a = np.asarray(a)
    if a.dtype == np.uint32:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int32)).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def route_inputs(wl):
    return (dev_i32(wl.req), torch.tensor([wl.T_valid], dtype=torch.int32, device="cuda"),
            dev_i32(np.asarray(wl.sub, np.uint32)))


def gpu_route(px, wl):
    rt = px.Route(wl.T_max, wl.n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    req, tv, sub = route_inputs(wl)
    px.xmix_route_build(req, tv, sub, rt, err)
    return rt, err


class Apps:
    """Device buffers of a workload's SAE apps: packed dictionaries, folded
    biases (every other app without one, so the batched call folds it),
    outputs, workspaces and, on every third app, a ring."""

    def __init__(self, px, wl, fold_every=2, ring_every=3):
        self.px, self.wl = px, wl
        self.items = []
        for i, s in enumerate(wl.layers[0].saes):
            W = px.xmix_sae_pack_encoder(dev_bits(s.W_enc))
            be, bd = dev_bits(s.b_enc), dev_bits(s.b_dec)
            c = None
            if i % fold_every == 0:
                c = torch.empty(s.m, dtype=torch.float32, device="cuda")
                px.xmix_sae_fold_bias(W, be, bd, c)
            ws = torch.empty(px.sae_encode_workspace(wl.T_max, wl.d, s.m, s.k),
                             dtype=torch.uint8, device="cuda")
            ring = px.Ring(97, 16 + 6 * s.k) if i % ring_every == 1 else None
            self.items.append(dict(s=s, W=W, be=be, bd=bd, c=c, ws=ws, ring=ring))
        self.reset()

    def reset(self):
        for it in self.items:
            k = it["s"].k
            it["idx"] = torch.full((self.wl.T_max, k), -7, dtype=torch.int32, device="cuda")
            it["val"] = torch.zeros((self.wl.T_max, k), dtype=torch.bfloat16, device="cuda")
            if it["ring"] is not None:
                it["ring"].slots.zero_()
                it["ring"].head.fill_(5)  # a head that is not at a slot boundary
                it["ring"].head[1] = 0

    def multi_apps(self):
        return [self.px.SaeApp(it["s"].bit, it["W"], it["be"], it["bd"], it["c"], it["s"].k,
                               it["idx"], it["val"], it["ws"], it["ring"], 100 + it["s"].bit)
                for it in self.items]

    def one_call_per_app(self, h, rt, req):
        for it in self.items:
            s = it["s"]
            if it["ring"] is None:
                self.px.xmix_sae_encode_topk(h, rt, s.bit, it["W"], it["be"], it["bd"], it["c"],
                                             s.k, it["idx"], it["val"], it["ws"])
            else:
                self.px.xmix_sae_encode_topk_ring(h, rt, s.bit, it["W"], it["be"], it["bd"],
                                                  it["c"], s.k, it["idx"], it["val"], it["ws"],
                                                  req, 3, 100 + s.bit, it["ring"])

    def results(self):
        torch.cuda.synchronize()
        out = []
        for it in self.items:
            r = it["ring"]
            out.append((it["idx"].cpu().numpy(), torch_bits(it["val"]),
                        None if r is None else (r.slots.cpu().numpy(), r.head.cpu().numpy())))
        return out


def assert_same(a, b):
    for (i1, v1, r1), (i2, v2, r2) in zip(a, b):
        assert np.array_equal(i1, i2)
        assert np.array_equal(v1, v2)
        assert (r1 is None) == (r2 is None)
        if r1 is not None:
            assert np.array_equal(r1[0], r2[0]) and np.array_equal(r1[1], r2[1])


def small_c5(T=256, n_clamp_apps=10, m=4096, seed=3):
    # 4 steering, 2 probe and n_clamp_apps SAE apps; two dictionary sizes
    return synth.make("c5", d=1024, T=T, m=m, k=32, p=0.3, n_steer=4, n_probe=2,
                      n_clamp_apps=n_clamp_apps, seed=seed)


@pytest.mark.parametrize("n_apps", [3, 10])
def test_encode_multi_matches_one_call_per_app(px, n_apps):
    """3 apps: one batched launch; 10 apps: two (at most 8 per launch)."""
    wl = small_c5(n_clamp_apps=n_apps)
    rt, err = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req = dev_i32(wl.req)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    apps.reset()
    px.xmix_sae_encode_topk_multi(h, rt, apps.multi_apps(), req, 3)
    assert_same(apps.results(), ref)
    # one app against the oracle
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    s = wl.layers[0].saes[-1]
    toks = lists[s.bit, :cnt[s.bit]][:24]
    idx_ref, _, _, pre = oracle.sae_encode(wl.layers[0].h, toks, s.W_enc, s.b_enc, s.b_dec, s.k,
                                           want_pre=True)
    idx, val, _ = ref[-1]
    for q, t in enumerate(toks):
        check_topk(idx[t], val[t], idx_ref[q], pre[q], s.k)
    # tokens without the app's bit are not written
    for it, (idx, _, _) in zip(apps.items, ref):
        b = it["s"].bit
        off = np.setdiff1d(np.arange(wl.T_max), lists[b, :cnt[b]])
        assert np.all(idx[off] == -7)


def test_routed_encode_multi_matches_route_build_then_multi(px):
    wl = small_c5(n_clamp_apps=5, seed=4)
    rt, err = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req, tv, sub = route_inputs(wl)
    apps = Apps(px, wl)
    px.xmix_sae_encode_topk_multi(h, rt, apps.multi_apps(), req, 3)
    ref = apps.results()
    ref_route = (rt.tok_mask.cpu().numpy(), rt.app_count.cpu().numpy(),
                 rt.app_tokens.cpu().numpy(), err.cpu().numpy())
    apps.reset()
    rt2 = px.Route(wl.T_max, wl.n_apps)
    rt2.tok_mask.fill_(-1)
    rt2.app_count.fill_(-1)
    rt2.app_tokens.fill_(-3)
    err2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_sae_encode_topk_multi(req, tv, sub, rt2, err2, h, apps.multi_apps(), 3)
    assert_same(apps.results(), ref)
    got_route = (rt2.tok_mask.cpu().numpy(), rt2.app_count.cpu().numpy(),
                 rt2.app_tokens.cpu().numpy(), err2.cpu().numpy())
    for a, b in zip(got_route, ref_route):
        assert np.array_equal(a, b)


def test_encode_multi_with_dictionaries_of_two_sizes(px):
    """Apps whose tiles differ in number follow each other in one launch."""
    wl = small_c5(n_clamp_apps=4, seed=5)
    big = small_c5(n_clamp_apps=4, m=8192, seed=6)
    saes = wl.layers[0].saes
    saes[1], saes[3] = big.layers[0].saes[1], big.layers[0].saes[3]
    rt, _ = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req = dev_i32(wl.req)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    apps.reset()
    px.xmix_sae_encode_topk_multi(h, rt, apps.multi_apps(), req, 3)
    assert_same(apps.results(), ref)


def test_encode_multi_prefill_shape_runs_apps_in_turn(px):
    """From 1025 token slots the apps run one after the other (the GEMM
    path); the results are those of one call per app."""
    wl = small_c5(T=1100, n_clamp_apps=2, seed=7)
    rt, _ = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req = dev_i32(wl.req)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    apps.reset()
    px.xmix_sae_encode_topk_multi(h, rt, apps.multi_apps(), req, 3)
    assert_same(apps.results(), ref)


def test_clamp_multi_matches_one_call_per_app(px):
    wl = small_c5(n_clamp_apps=10, seed=8)
    rt, _ = gpu_route(px, wl)
    h0 = dev_bits(wl.layers[0].h)
    req = dev_i32(wl.req)
    apps = Apps(px, wl, ring_every=10 ** 6)
    px.xmix_sae_encode_topk_multi(h0, rt, apps.multi_apps(), req, 3)
    torch.cuda.synchronize()
    clamp = []
    for i, it in enumerate(apps.items):
        s = it["s"]
        ids = dev_i32(s.clamp_ids)
        vals = torch.from_numpy(np.asarray(s.clamp_vals, np.float32) * (1 + i)).cuda()
        clamp.append((s.bit, it["idx"], it["val"], dev_bits(s.W_dec), ids, vals))
    # reference: one call per app, in order, each with its own delta
    h_ref = h0.clone()
    d_ref = [torch.zeros((wl.T_max, wl.d), dtype=torch.float32, device="cuda") for _ in clamp]
    for c, dref in zip(clamp, d_ref):
        px.xmix_sae_clamp_decode(h_ref, rt, *c, delta_out=dref)
    h = h0.clone()
    d_got = [torch.zeros_like(x) for x in d_ref]
    px.xmix_sae_clamp_decode_multi(h, rt, [c + (dg,) for c, dg in zip(clamp, d_got)])
    torch.cuda.synchronize()
    assert np.array_equal(torch_bits(h), torch_bits(h_ref))
    for a, b in zip(d_got, d_ref):
        assert torch.equal(a, b)
    # rows of tokens with no clamp app are untouched
    tm, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    bits = sum(1 << c[0] for c in clamp)
    untouched = (tm & np.uint32(bits)) == 0
    assert np.array_equal(torch_bits(h)[untouched], wl.layers[0].h[untouched])
    # the order of the apps matters only through the roundings: the reverse
    # order, one call per app, matches the batched call in reverse order
    h_rev_ref = h0.clone()
    for c in reversed(clamp):
        px.xmix_sae_clamp_decode(h_rev_ref, rt, *c)
    h_rev = h0.clone()
    px.xmix_sae_clamp_decode_multi(h_rev, rt, list(reversed(clamp)))
    torch.cuda.synchronize()
    assert np.array_equal(torch_bits(h_rev), torch_bits(h_rev_ref))


def test_encode_multi_workgroups_run_many_slices_and_skip_empty_apps(px):
    """Eight apps of 256 slices each on the persistent grid: every
    workgroup runs several slices, one after the other, over up to four
    token tiles each, and two apps without a subscriber are skipped."""
    wl = small_c5(T=512, n_clamp_apps=8, m=65536, seed=9)
    wl.sub = (wl.sub | np.uint32(0xFF << 6)).astype(np.uint32)  # every request: every SAE
    saes = wl.layers[0].saes
    for s in (saes[2], saes[5]):
        wl.sub &= ~np.uint32(1 << s.bit)
    sparse = saes[6].bit  # one app with few tokens: one token tile
    wl.sub[np.arange(len(wl.sub)) % 7 != 0] &= ~np.uint32(1 << sparse)
    rt, _ = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req = dev_i32(wl.req)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    apps.reset()
    px.xmix_sae_encode_topk_multi(h, rt, apps.multi_apps(), req, 3)
    got = apps.results()
    assert_same(got, ref)
    # the routed form as well
    apps.reset()
    rt2 = px.Route(wl.T_max, wl.n_apps)
    err2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    r, tv, sb = route_inputs(wl)
    px.xmix_route_sae_encode_topk_multi(r, tv, sb, rt2, err2, h, apps.multi_apps(), 3)
    assert_same(apps.results(), ref)
    assert np.array_equal(rt2.app_count.cpu().numpy(), rt.app_count.cpu().numpy())
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    assert cnt[saes[2].bit] == 0 and cnt[saes[5].bit] == 0 and cnt[saes[0].bit] == 512
    # the empty apps' outputs are untouched
    for j in (2, 5):
        assert np.all(got[j][0] == -7)
    # tokens of every token tile of one app against the oracle
    s = saes[3]
    toks = lists[s.bit, :cnt[s.bit]][[0, 127, 128, 300, 383, 384, 511]]
    idx_ref, _, _, pre = oracle.sae_encode(wl.layers[0].h, toks, s.W_enc, s.b_enc, s.b_dec, s.k,
                                           want_pre=True)
    idx, val, _ = got[3]
    for q, t in enumerate(toks):
        check_topk(idx[t], val[t], idx_ref[q], pre[q], s.k)


def test_encode_multi_between_decode_and_prefill_shapes(px):
    """513 to 1024 token slots: the batched launch over the apps' blocked
    tile grids (neither the persistent grid nor the prefill GEMM)."""
    wl = small_c5(T=700, n_clamp_apps=3, seed=10)
    rt, _ = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req = dev_i32(wl.req)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    apps.reset()
    px.xmix_sae_encode_topk_multi(h, rt, apps.multi_apps(), req, 3)
    assert_same(apps.results(), ref)


def test_routed_encode_multi_publishes_the_routing_without_subscribers(px):
    """No request subscribes to anything: the routed batched call still
    publishes every app's (empty) list, count and mask, as the route build
    does, and writes no output row."""
    wl = small_c5(n_clamp_apps=4, seed=11)
    wl.sub = np.zeros_like(wl.sub)
    rt, err = gpu_route(px, wl)
    ref = (rt.tok_mask.cpu().numpy(), rt.app_count.cpu().numpy(), rt.app_tokens.cpu().numpy(),
           err.cpu().numpy())
    h = dev_bits(wl.layers[0].h)
    req, tv, sub = route_inputs(wl)
    apps = Apps(px, wl)
    rt2 = px.Route(wl.T_max, wl.n_apps)
    rt2.tok_mask.fill_(-1)
    rt2.app_count.fill_(-1)
    rt2.app_tokens.fill_(-3)
    err2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_sae_encode_topk_multi(req, tv, sub, rt2, err2, h, apps.multi_apps(), 3)
    got = (rt2.tok_mask.cpu().numpy(), rt2.app_count.cpu().numpy(),
           rt2.app_tokens.cpu().numpy(), err2.cpu().numpy())
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)
    for idx, _, ring in apps.results():
        assert np.all(idx == -7)
        if ring is not None:
            assert np.all(ring[0] == 0) and ring[1][0] == 5


def test_routed_encode_multi_with_fewer_slices_than_apps(px):
    """Three one-slice dictionaries (m = 256) among 9 apps: the persistent
    grid has more workgroups than slices, so that every app's list is
    published; the results are those of one call per app."""
    wl = small_c5(n_clamp_apps=3, m=256, seed=12)
    rt, err = gpu_route(px, wl)
    h = dev_bits(wl.layers[0].h)
    req, tv, sub = route_inputs(wl)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    ref_route = (rt.tok_mask.cpu().numpy(), rt.app_count.cpu().numpy(),
                 rt.app_tokens.cpu().numpy(), err.cpu().numpy())
    apps.reset()
    rt2 = px.Route(wl.T_max, wl.n_apps)
    rt2.app_count.fill_(-1)
    rt2.app_tokens.fill_(-3)
    err2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_sae_encode_topk_multi(req, tv, sub, rt2, err2, h, apps.multi_apps(), 3)
    assert_same(apps.results(), ref)
    got = (rt2.tok_mask.cpu().numpy(), rt2.app_count.cpu().numpy(),
           rt2.app_tokens.cpu().numpy(), err2.cpu().numpy())
    for a, b in zip(got, ref_route):
        assert np.array_equal(a, b)


def test_routed_encode_multi_with_mixed_k_padding_and_t_valid(px):
    """Apps with k = 8, 32 and 64 in one batch (each its own candidate cap
    and threshold quantile), a padded slot, a request id out of range and
    T_valid below T_max: the routed batched call matches the route build
    followed by one call per app, error word included."""
    wl = small_c5(T=300, n_clamp_apps=3, seed=13)
    saes = wl.layers[0].saes
    for s, k in zip(saes, (8, 32, 64)):
        s.k = k
    wl.req = wl.req.copy()
    wl.req[5] = -1              # padding
    wl.req[7] = wl.R_max + 3    # out of range: routes nowhere, flags the error word
    wl.T_valid = 290
    rt, err = gpu_route(px, wl)
    assert int(err.item()) != 0
    h = dev_bits(wl.layers[0].h)
    req, tv, sub = route_inputs(wl)
    apps = Apps(px, wl)
    apps.one_call_per_app(h, rt, req)
    ref = apps.results()
    ref_route = (rt.tok_mask.cpu().numpy(), rt.app_count.cpu().numpy(),
                 rt.app_tokens.cpu().numpy(), err.cpu().numpy())
    apps.reset()
    rt2 = px.Route(wl.T_max, wl.n_apps)
    err2 = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_sae_encode_topk_multi(req, tv, sub, rt2, err2, h, apps.multi_apps(), 3)
    assert_same(apps.results(), ref)
    got = (rt2.tok_mask.cpu().numpy(), rt2.app_count.cpu().numpy(),
           rt2.app_tokens.cpu().numpy(), err2.cpu().numpy())
    for a, b in zip(got, ref_route):
        assert np.array_equal(a, b)
    # the k = 64 app against the oracle
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    s = saes[2]
    toks = lists[s.bit, :cnt[s.bit]][::9]
    idx_ref, _, _, pre = oracle.sae_encode(wl.layers[0].h, toks, s.W_enc, s.b_enc, s.b_dec, s.k,
                                           want_pre=True)
    idx, val, _ = ref[2]
    for q, t in enumerate(toks):
        check_topk(idx[t], val[t], idx_ref[q], pre[q], s.k)
