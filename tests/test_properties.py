"""Property tests (hypothesis, small shapes): routing invariants of the
oracle on the CPU, and GPU routing, steering, readback and SAE encode
against the oracle on generated batches (padding, bad ids, ragged T_valid,
any mask; for the encode both kernel paths and dictionaries drawn from
several distributions)."""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle


@st.composite
def batches(draw, max_T=300, max_R=12):
    T = draw(st.integers(1, max_T))
    R = draw(st.integers(1, max_R))
    n_apps = draw(st.integers(1, 32))
    req = np.array(draw(st.lists(st.integers(-3, R + 2), min_size=T, max_size=T)), np.int32)
    sub = np.array(draw(st.lists(st.integers(0, 2**32 - 1), min_size=R, max_size=R)), np.uint32)
    T_valid = draw(st.integers(-2, T + 2))
    return T, R, n_apps, req, sub, T_valid


@settings(max_examples=60, deadline=None, derandomize=True)
@given(batches())
def test_oracle_route_invariants(b):
    T, R, n_apps, req, sub, T_valid = b
    tm, cnt, lists, err = oracle.route(req, T_valid, sub, n_apps)
    keep = np.uint32((1 << n_apps) - 1) if n_apps < 32 else np.uint32(0xFFFFFFFF)
    tv = min(max(T_valid, 0), T)
    # masks: the request's subscription restricted to the registered apps
    for t in range(T):
        r = req[t]
        want = sub[r] & keep if (t < tv and 0 <= r < R) else 0
        assert tm[t] == want
    # counts, strictly increasing lists that list exactly the tokens with the bit
    pops = sum(bin(int(x)).count("1") for x in tm)
    assert int(cnt.sum()) == pops
    for a in range(n_apps):
        L = lists[a, :cnt[a]]
        assert np.all(np.diff(L) > 0)
        assert set(L.tolist()) == {t for t in range(T) if (tm[t] >> a) & 1}
        assert np.all(lists[a, cnt[a]:] == -1)
    # error bits
    bad_req = any(req[t] >= R for t in range(tv))
    assert bool(err & 1) == bad_req
    assert bool(err & 2) == (T_valid < 0 or T_valid > T)


@pytest.mark.gpu
@settings(max_examples=25, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])
@given(batches(max_T=2100))
def test_gpu_route_matches_oracle(b):
    import torch
    import paper_2607_22595_amd as px
    T, R, n_apps, req, sub, T_valid = b
    rt = px.Route(T, n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_build(torch.from_numpy(req).cuda(),
                        torch.tensor([T_valid], dtype=torch.int32, device="cuda"),
                        torch.from_numpy(sub.view(np.int32)).cuda(), rt, err)
    torch.cuda.synchronize()
    tm, cnt, lists, e = oracle.route(req, T_valid, sub, n_apps)
    assert np.array_equal(rt.tok_mask.cpu().numpy().view(np.uint32), tm)
    assert np.array_equal(rt.app_count.cpu().numpy(), cnt)
    assert np.array_equal(rt.app_tokens.cpu().numpy(), lists)
    assert int(err.item()) == e


@pytest.mark.gpu
@settings(max_examples=20, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])
@given(batches(max_T=600, max_R=8), st.integers(1, 4), st.sampled_from([256, 264, 1024]),
       st.integers(0, 2**31 - 1))
def test_gpu_steer_matches_oracle(b, n_steer, d, seed):
    import torch
    import paper_2607_22595_amd as px
    import synth
    from parity import check_steer, torch_bits
    T, R, n_apps, req, sub, T_valid = b
    n_apps = max(n_apps, n_steer)
    h = synth.normal_bf16(f"prop/h/{seed}", (T, d), 1.0)
    v = synth.normal_bf16(f"prop/v/{seed}", (n_steer, d), 1.0 / np.sqrt(d))
    alpha = synth.uniform_f32(f"prop/a/{seed}", (R, n_steer), -8.0, 8.0)
    bits = list(range(n_steer))
    rt = px.Route(T, n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    req_d = torch.from_numpy(req).cuda()
    px.xmix_route_build(req_d, torch.tensor([T_valid], dtype=torch.int32, device="cuda"),
                        torch.from_numpy(sub.view(np.int32)).cuda(), rt, err)
    hd = torch.from_numpy(h.view(np.int16)).cuda().view(torch.bfloat16)
    vd = torch.from_numpy(v.view(np.int16)).cuda().view(torch.bfloat16)
    px.xmix_steer_apply(hd, rt, req_d, vd, bits, torch.from_numpy(alpha).cuda())
    torch.cuda.synchronize()
    tm, _, _, _ = oracle.route(req, T_valid, sub, n_apps)
    ref = oracle.steer(h, tm, req, v, bits, alpha)
    rows = (tm & np.uint32(sum(1 << x for x in bits))) != 0
    check_steer(torch_bits(hd), ref, h, rows, True)


@pytest.mark.gpu
@settings(max_examples=20, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])
@given(batches(max_T=700, max_R=8), st.integers(1, 300), st.integers(0, 3),
       st.integers(0, 2**40))
def test_gpu_readback_matches_oracle(b, cap, calls, head0):
    import torch
    import paper_2607_22595_amd as px
    T, R, n_apps, req, sub, T_valid = b
    rows = np.arange(T * 8, dtype=np.int32).reshape(T, 8) * 7 + 3
    rt = px.Route(T, n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    req_d = torch.from_numpy(req).cuda()
    px.xmix_route_build(req_d, torch.tensor([T_valid], dtype=torch.int32, device="cuda"),
                        torch.from_numpy(sub.view(np.int32)).cuda(), rt, err)
    tm, _, _, _ = oracle.route(req, T_valid, sub, n_apps)
    app = n_apps - 1
    ring = px.Ring(cap, 16 + 32)
    ring.head[0] = head0
    slots = np.zeros((cap, 48), np.uint8)
    head = head0
    rows_d = torch.from_numpy(rows).cuda()
    for _ in range(calls + 1):
        px.xmix_readback_compact([rows_d], rt, app, req_d, 2, app, ring)
        slots, head = oracle.compact([rows.view(np.uint8).reshape(T, -1)], tm, app, req, 2, app,
                                     slots, head)
    torch.cuda.synchronize()
    assert int(ring.head[0].item()) == head and int(ring.head[1].item()) == 0
    assert np.array_equal(ring.slots.cpu().numpy(), slots)


# ------------------------------------------------------------ SAE encode

@st.composite
def encode_cases(draw):
    """A decode-kernel batch (up to 300 slots) or a prefill-GEMM batch (1025
    slots and more), with dictionaries drawn from several distributions:
    Gaussian rows; rows scaled by Pareto(1.5) or log-normal factors (norms
    that differ by orders of magnitude); widely spread biases; exact ties
    (duplicated rows); and a cluster of rows along one direction the tokens
    share, packed into a few slices (winners crowding one slice)."""
    d = draw(st.sampled_from([256, 512]))
    decode = draw(st.booleans())
    m = draw(st.sampled_from([256, 512, 1024, 4096, 16384] if decode else [256, 1024, 4096]))
    k = draw(st.integers(1, min(64, m)))
    T = draw(st.integers(1, 300)) if decode else draw(st.integers(1025, 1100))
    n_sub = draw(st.integers(0, T))
    kind = draw(st.sampled_from(["gaussian", "pareto", "lognormal", "bias", "ties", "cluster"]))
    seed = draw(st.integers(0, 1000))
    return d, m, k, T, n_sub, kind, seed


def _dictionary(sae, d, kind, seed):
    import synth
    from parity import bf16_f64

    def bits(a):
        import torch
        return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16) \
            .view(torch.int16).numpy().view(np.uint16)
    m = sae.m
    W = bf16_f64(sae.W_enc).reshape(m, d)
    b = bf16_f64(sae.b_enc)
    u = synth.uniform01(f"prop/{kind}", m, seed=seed)
    if kind == "pareto":
        W *= np.minimum((1.0 - u) ** (-1.0 / 1.5), 200.0)[:, None]
    elif kind == "lognormal":
        W *= np.exp(1.5 * bf16_f64(synth.normal_bf16(f"prop/ln", (m,), 1.0, seed=seed)))[:, None]
    elif kind == "bias":
        b = 3.0 * bf16_f64(synth.normal_bf16("prop/bias", (m,), 1.0, seed=seed)) - 1.0
    elif kind == "ties":
        src = (u * m).astype(np.int64) % m
        dst = np.nonzero(u < 0.05)[0]
        W[dst] = W[src[dst]]
        b[dst] = b[src[dst]]
    elif kind == "cluster":
        v = bf16_f64(synth.normal_bf16("prop/dir", (d,), 1.0, seed=seed))
        v /= np.linalg.norm(v)
        rows = np.nonzero((np.arange(m) // 256 < 2) & (u < 0.25))[0]
        W[rows] = (3.0 + u[rows, None]) * v[None, :] / np.sqrt(d) * 4.0
    sae.W_enc = bits(W)
    sae.b_enc = bits(b)
    return v if kind == "cluster" else None


@pytest.mark.gpu
@settings(max_examples=60, deadline=None, derandomize=True,
          suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])
@given(encode_cases())
def test_gpu_encode_matches_oracle(case):
    import torch
    import paper_2607_22595_amd as px
    import synth
    from parity import bf16_f64, check_topk, torch_bits
    d, m, k, T, n_sub, kind, seed = case
    wl = synth.make("c3", d=d, m=m, k=k, T=T, n_sub=n_sub, seed=seed)
    sae = wl.layers[0].saes[0]
    v = _dictionary(sae, d, kind, seed)
    h = wl.layers[0].h
    if v is not None:  # the tokens share the cluster's direction
        h = torch.from_numpy((bf16_f64(h) + 2.0 * np.sqrt(d) * v[None, :]).astype(np.float32)) \
            .to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    tm, cnt, lists, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    toks = lists[0, :cnt[0]]
    rt = px.Route(T, wl.n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_build(torch.from_numpy(wl.req).cuda(),
                        torch.tensor([wl.T_valid], dtype=torch.int32, device="cuda"),
                        torch.from_numpy(wl.sub.view(np.int32)).cuda(), rt, err)

    def dev(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda() \
            .view(torch.bfloat16)
    W = px.xmix_sae_pack_encoder(dev(sae.W_enc))
    be, bd = dev(sae.b_enc), dev(sae.b_dec)
    c = torch.empty(m, dtype=torch.float32, device="cuda")
    px.xmix_sae_fold_bias(W, be, bd, c)
    idx = torch.full((T, k), -7, dtype=torch.int32, device="cuda")
    val = torch.zeros((T, k), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(px.sae_encode_workspace(T, d, m, k), dtype=torch.uint8, device="cuda")
    px.xmix_sae_encode_topk(dev(h), rt, sae.bit, W, be, bd, c, k, idx, val, ws)
    torch.cuda.synchronize()
    idx, val = idx.cpu().numpy(), torch_bits(val)
    if len(toks):
        idx_ref, _, _, pre = oracle.sae_encode(h, toks, sae.W_enc, sae.b_enc, sae.b_dec, k,
                                               want_pre=True)
        for q, t in enumerate(toks):
            check_topk(idx[t], val[t], idx_ref[q], pre[q], k)
    off = np.setdiff1d(np.arange(T), toks)
    assert np.all(idx[off] == -7)
