"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test checks an oracle function against something fixed independently:
a hand-derived value, a closed form, a library routine on a special case,
an invariant, or brute force on a tiny input.  The cases are chosen so that
a plausible slip (a dropped term, a wrong sign or index, a transposed
operand, a wrong tie rule) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def f32_to_bf16_torch(x):
    """Library RNE: torch's fp32 -> bf16 conversion, exact for fp32 inputs."""
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_vals(bits):
    return synth.bf16_bits_to_f32(bits).astype(np.float64)


# ------------------------------------------------------------------ rounding

def test_round_bf16_golden_cases():
    """Hand-derived RNE cases (bf16 = 1 sign, 8 exponent, 7 fraction bits)."""
    path = os.path.join(GOLDEN, "bf16_rne.txt")
    n = 0
    with open(path) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            xs, bits = line.split()
            assert oracle.round_bf16(float.fromhex(xs)) == int(bits, 16), xs
            n += 1
    assert n >= 10


def test_round_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(7)
    x = np.concatenate([rng.standard_normal(5000) * s for s in (1e-3, 1.0, 1e3)]).astype(np.float32)
    got = np.array([oracle.round_bf16(float(v)) for v in x], np.uint16)
    assert np.array_equal(got, f32_to_bf16_torch(x))


def test_round_bf16_rounds_once_from_double():
    # 1 + 2^-8 + 2^-40 is just above the tie: a detour through fp32 would
    # land exactly on the tie and round down to even; direct rounding goes up.
    x = 1.0 + 2.0 ** -8 + 2.0 ** -40
    assert oracle.round_bf16(x) == 0x3F81


# ------------------------------------------------------------------- routing

def brute_route(req, T_valid, sub, n_apps):
    T = len(req)
    R = len(sub)
    err = 0
    tv = T_valid
    if tv < 0 or tv > T:
        err |= 2
        tv = min(max(tv, 0), T)
    mask = []
    for t in range(T):
        m = 0
        if t < tv:
            r = int(req[t])
            if r >= R:
                err |= 1
            elif r >= 0:
                m = int(sub[r]) & ((1 << n_apps) - 1)
        mask.append(m)
    lists = [[t for t in range(T) if (mask[t] >> a) & 1] for a in range(n_apps)]
    return mask, lists, err


@pytest.mark.parametrize("seed", range(6))
def test_route_brute_force(seed):
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 200))
    R = int(rng.integers(1, 40))
    n_apps = int(rng.integers(1, 33))
    req = rng.integers(-2, R + 3, size=T).astype(np.int32)
    sub = rng.integers(0, 2 ** 32, size=R, dtype=np.uint64).astype(np.uint32)
    T_valid = int(rng.integers(-1, T + 2))
    tok_mask, count, app_tokens, err = oracle.route(req, T_valid, sub, n_apps)
    mask, lists, berr = brute_route(req, T_valid, sub, n_apps)
    assert tok_mask.tolist() == mask
    assert err == berr
    for a in range(n_apps):
        assert count[a] == len(lists[a])
        assert app_tokens[a, :count[a]].tolist() == lists[a]
        assert np.all(app_tokens[a, count[a]:] == -1)
    # invariants
    assert count.sum() == sum(bin(m).count("1") for m in mask)


def test_route_all_subscribed_lists_every_token():
    T, R = 50, 50
    req = np.arange(T, dtype=np.int32)
    sub = np.full(R, 0xFFFFFFFF, np.uint32)
    tok_mask, count, app_tokens, err = oracle.route(req, T, sub, 32)
    assert err == 0 and np.all(count == T)
    assert np.all(app_tokens == np.arange(T)[None, :])


# ------------------------------------------------------------------ steering

def test_steer_alpha_zero_is_identity(synth):
    wl = synth.make("c2", d=256, T=32, n_layers=1)
    L = wl.layers[0]
    tok_mask, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    v = np.stack([s.v for s in L.steer])
    alpha = np.zeros_like(wl.alpha)
    out = oracle.steer(L.h, tok_mask, wl.req, v, [s.bit for s in L.steer], alpha)
    assert np.array_equal(bf16_vals(out), bf16_vals(L.h))


def test_steer_one_hot_changes_one_channel():
    d, T = 64, 8
    h = synth.normal_bf16("pin/steer/h", (T, d), 1.0)
    v = np.zeros((1, d), np.uint16)
    v[0, 5] = 0x3F80  # 1.0
    alpha = np.array([[0.75], [-3.0]] * 4, np.float32)
    req = np.arange(T, dtype=np.int32)
    tok_mask = np.array([1, 0] * 4, np.uint32)
    out = oracle.steer(h, tok_mask, req, v, [0], alpha)
    hv = bf16_vals(h)
    ov = bf16_vals(out)
    for t in range(T):
        if tok_mask[t]:
            other = [i for i in range(d) if i != 5]
            assert np.array_equal(ov[t, other], hv[t, other])
            exact = np.float32(hv[t, 5] + alpha[t, 0])  # exact in fp32
            assert out[t, 5] == f32_to_bf16_torch([exact])[0]
        else:
            assert np.array_equal(out[t], h[t])


def test_steer_sums_vectors_exactly():
    """Several subscribed vectors are summed and rounded once.  The inputs are
    dyadic with a narrow exponent range, so the exact sum is an fp32 value
    and torch's fp32->bf16 rounding gives the expected bits."""
    rng = np.random.default_rng(3)
    d, T, n_s = 32, 12, 3
    h = f32_to_bf16_torch(rng.integers(-64, 64, (T, d)) / 16.0)
    v = f32_to_bf16_torch(rng.integers(-64, 64, (n_s, d)) / 64.0)
    alpha = rng.integers(-8, 9, (T, n_s)).astype(np.float32)
    req = np.arange(T, dtype=np.int32)
    tok_mask = rng.integers(0, 8, T).astype(np.uint32)
    out = oracle.steer(h, tok_mask, req, v, [0, 1, 2], alpha)
    hv, vv = bf16_vals(h), bf16_vals(v)
    for t in range(T):
        if tok_mask[t] == 0:
            assert np.array_equal(out[t], h[t])
            continue
        acc = hv[t].copy()
        for s in range(n_s):
            if (tok_mask[t] >> s) & 1:
                acc = acc + alpha[t, s] * vv[s]
        assert np.array_equal(acc.astype(np.float32).astype(np.float64), acc)  # exact
        assert np.array_equal(out[t], f32_to_bf16_torch(acc))


def test_steer_sign_and_app_bit_mapping():
    # vector s is gated by bit app_bits[s], not by bit s
    d = 16
    h = np.zeros((2, d), np.uint16)
    v = f32_to_bf16_torch(np.ones((2, d)))
    alpha = np.array([[1.0, -2.0], [1.0, -2.0]], np.float32)
    out = oracle.steer(h, np.array([1 << 7, 1 << 3], np.uint32), np.array([0, 1], np.int32),
                       v, [3, 7], alpha)
    assert np.all(bf16_vals(out[0]) == -2.0)   # bit 7 -> vector 1, alpha -2
    assert np.all(bf16_vals(out[1]) == 1.0)    # bit 3 -> vector 0, alpha 1


def test_steer_fp32_storage():
    wl = synth.make("c1")
    L = wl.layers[0]
    tok_mask, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    out = oracle.steer(L.h, tok_mask, wl.req, L.steer[0].v[None], [0], wl.alpha)
    for t in range(wl.T_max):
        if tok_mask[t] & 1:
            exp = (L.h[t].astype(np.float64) + 4.0 * L.steer[0].v.astype(np.float64)).astype(np.float32)
            assert np.array_equal(out[t], exp)
        else:
            assert np.array_equal(out[t], L.h[t])


# -------------------------------------------------------------------- probes

def test_probe_matches_fsum_dot():
    wl = synth.make("c2", d=512, T=16, n_layers=1)
    L = wl.layers[0]
    tok_mask, _, _, _ = oracle.route(wl.req, wl.T_valid, wl.sub, wl.n_apps)
    w = np.stack([p.w for p in L.probes])
    b = np.array([p.b for p in L.probes], np.float32)
    bits = [p.bit for p in L.probes]
    logit, score = oracle.probe_token(L.h, tok_mask, w, b, bits)
    hv, wv = bf16_vals(L.h), bf16_vals(w)
    n_checked = 0
    for p in range(len(bits)):
        for t in range(wl.T_max):
            if (tok_mask[t] >> bits[p]) & 1:
                ref = math.fsum([float(b[p])] + [wv[p, i] * hv[t, i] for i in range(wl.d)])
                assert abs(logit[p, t] - ref) <= 1e-12 * math.fsum(abs(wv[p, i] * hv[t, i]) for i in range(wl.d))
                assert score[p, t] == pytest.approx(1 / (1 + math.exp(-ref)), rel=1e-14)
                n_checked += 1
            else:
                assert np.isnan(logit[p, t])
    assert n_checked > 0


def test_probe_closed_forms():
    d = 64
    h = synth.normal_bf16("pin/probe/h", (4, d), 1.0)
    w = np.zeros((2, d), np.uint16)
    w[0, 9] = 0x3F80          # e_9
    b = np.array([0.25, 0.0], np.float32)
    logit, score = oracle.probe_token(h, np.full(4, 3, np.uint32), w, b, [0, 1])
    assert np.array_equal(logit[0], bf16_vals(h[:, 9]) + 0.25)
    assert np.all(logit[1] == 0.0) and np.all(score[1] == 0.5)


def test_probe_logistic_closed_forms():
    """The score's orientation and scale, from values whose logistic is known
    in closed form: sigma(ln 3) = 3/4, sigma(-ln 3) = 1/4, sigma(ln 9) = 9/10,
    sigma(0) = 1/2 and sigma(-x) = 1 - sigma(x).  A probe with w = e_0 and
    b = 0 on fp32 rows makes the logit exactly the row's first value."""
    d = 8
    xs = np.array([math.log(3.0), -math.log(3.0), math.log(9.0), 0.0, 2.5, -2.5, 17.0, -17.0],
                  np.float32)
    h = np.zeros((xs.size, d), np.float32)
    h[:, 0] = xs
    w = np.zeros((1, d), np.float32)
    w[0, 0] = 1.0
    logit, score = oracle.probe_token(h, np.ones(xs.size, np.uint32), w,
                                      np.zeros(1, np.float32), [0])
    assert np.array_equal(logit[0], xs.astype(np.float64))
    # float32(ln 3) differs from ln 3 by < 2^-24 relative; sigma' <= 1/4
    assert abs(score[0, 0] - 0.75) <= 1e-7
    assert abs(score[0, 1] - 0.25) <= 1e-7
    assert abs(score[0, 2] - 0.9) <= 1e-7
    assert score[0, 3] == 0.5
    assert score[0, 4] + score[0, 5] == pytest.approx(1.0, abs=1e-15)
    assert score[0, 4] > 0.5 > score[0, 5]
    assert score[0, 6] + score[0, 7] == pytest.approx(1.0, abs=1e-15)
    assert 1.0 - score[0, 6] == pytest.approx(math.exp(-17.0) / (1 + math.exp(-17.0)),
                                              rel=1e-6)


def test_probe_mean_pins():
    d, R = 32, 4
    lens = [1, 3, 0, 5]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    h = synth.normal_bf16("pin/pool/h", (T, d), 1.0)
    h[1:4] = h[1]               # request 1: three identical rows
    w = synth.normal_bf16("pin/pool/w", (1, d), 0.2)
    b = np.array([0.1], np.float32)
    tok_mask = np.full(T, 1, np.uint32)
    tok_mask[cu[3]:cu[4]] = 0   # request 3 unsubscribed
    lt, st = oracle.probe_token(h, tok_mask | 1, w, b, [0])
    lm, sm = oracle.probe_mean(h, tok_mask, w, b, [0], cu)
    assert lm[0, 0] == lt[0, 0]                     # single-token request
    assert lm[0, 1] == pytest.approx(lt[0, 1], rel=1e-14, abs=1e-15)  # identical rows
    assert np.isnan(lm[0, 2]) and np.isnan(lm[0, 3])  # empty / unsubscribed
    hv, wv = bf16_vals(h), bf16_vals(w)
    ref = float(np.float32(0.1)) + math.fsum(wv[0, i] * hv[t, i] for t in range(1, 4) for i in range(d)) / 3
    assert lm[0, 1] == pytest.approx(ref, rel=1e-13)
    assert sm[0, 1] == pytest.approx(1 / (1 + math.exp(-lm[0, 1])), rel=1e-14)


def test_probe_last_pins():
    d = 24
    lens = [2, 1, 0, 4]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    T = int(cu[-1])
    h = synth.normal_bf16("pin/last/h", (T, d), 1.0)
    w = synth.normal_bf16("pin/last/w", (2, d), 0.3)
    b = np.array([0.25, -0.5], np.float32)
    tok_mask = np.full(T, 0b11, np.uint32)
    tok_mask[cu[3]:cu[4]] = 0b10  # request 3 has only the second probe's bit
    ll, sl = oracle.probe_last(h, tok_mask, w, b, [0, 1], cu)
    lt, st = oracle.probe_token(h, np.full(T, 0b11, np.uint32), w, b, [0, 1])
    # equals the per-token probe of each span's last token
    assert ll[0, 0] == lt[0, 1] and ll[1, 0] == lt[1, 1]
    assert ll[0, 1] == lt[0, 2]                         # single-token span
    assert np.isnan(ll[0, 2]) and np.isnan(ll[1, 2])    # empty span
    assert np.isnan(ll[0, 3]) and ll[1, 3] == lt[1, 6]  # per-probe subscription
    hv, wv = bf16_vals(h), bf16_vals(w)
    ref = float(np.float32(-0.5)) + math.fsum(wv[1, i] * hv[6, i] for i in range(d))
    assert ll[1, 3] == pytest.approx(ref, rel=1e-13)
    assert sl[1, 3] == pytest.approx(1 / (1 + math.exp(-ll[1, 3])), rel=1e-14)


# ------------------------------------------------------------- SAE encode

def sort_topk(pre, k):
    order = np.lexsort((np.arange(pre.size), -pre))  # value desc, index asc
    return order[:k]


@pytest.mark.parametrize("m,k", [(64, 1), (64, 8), (64, 64), (100, 8), (256, 1), (256, 256)])
def test_topk_matches_full_sort(m, k):
    rng = np.random.default_rng(m * 1000 + k)
    pre = rng.standard_normal(m)
    pre[rng.integers(0, m, m // 4)] = 0.5          # forced ties
    pre[rng.integers(0, m, m // 8)] = -1.25
    idx, ve, vb = oracle.topk(pre, k)
    exp = sort_topk(pre, k)
    assert idx.tolist() == exp.tolist()
    assert np.array_equal(ve, np.maximum(pre[exp], 0.0))
    # values that are exact in fp32 round the same way as torch's conversion
    relu32 = np.maximum(pre[exp], 0.0).astype(np.float32)
    exact = relu32.astype(np.float64) == np.maximum(pre[exp], 0.0)
    assert np.array_equal(vb[exact], f32_to_bf16_torch(relu32[exact]))


def test_topk_ties_take_lower_index_and_pad_with_zero_values():
    pre = np.array([-3.0, 2.0, -1.0, 2.0, -1.0, -5.0])
    idx, ve, vb = oracle.topk(pre, 5)
    assert idx.tolist() == [1, 3, 2, 4, 0]
    assert ve.tolist() == [2.0, 2.0, 0.0, 0.0, 0.0]
    assert vb.tolist() == [0x4000, 0x4000, 0, 0, 0]


def test_sae_identity_dictionary():
    """m = d, W_enc = I, b_enc = 0: pre = h - b_dec exactly."""
    d = 64
    h = synth.normal_bf16("pin/sae_id/h", (3, d), 1.0)
    b_dec = synth.normal_bf16("pin/sae_id/bdec", (d,), 0.1)
    W = np.zeros((d, d), np.uint16)
    W[np.arange(d), np.arange(d)] = 0x3F80
    b_enc = np.zeros(d, np.uint16)
    idx, val, ve, pre = oracle.sae_encode(h, [0, 1, 2], W, b_enc, b_dec, 8, want_pre=True)
    for q in range(3):
        u = bf16_vals(h[q]) - bf16_vals(b_dec)
        assert np.array_equal(pre[q], u)
        assert idx[q].tolist() == sort_topk(u, 8).tolist()


def test_sae_planted_features():
    """Rows planted along the token direction win with a known margin."""
    d, m, k = 128, 512, 4
    W = synth.normal_bf16("pin/sae_plant/W", (m, d), 0.01)
    h = synth.normal_bf16("pin/sae_plant/h", (1, d), 1.0)
    planted = [17, 300, 42, 511]
    for r, j in enumerate(planted):
        W[j] = f32_to_bf16_torch(bf16_vals(h[0]) * (1.0 - 0.1 * r) / d)
    zeros_m = np.zeros(m, np.uint16)
    zeros_d = np.zeros(d, np.uint16)
    idx, val, ve, pre = oracle.sae_encode(h, [0], W, zeros_m, zeros_d, k, want_pre=True)
    assert idx[0].tolist() == planted


def test_sae_gemm_matches_numpy_float64():
    d, m = 96, 200
    h = synth.normal_bf16("pin/sae_mm/h", (5, d), 1.0)
    W = synth.normal_bf16("pin/sae_mm/W", (m, d), 1 / np.sqrt(d))
    b_enc = synth.normal_bf16("pin/sae_mm/be", (m,), 0.1)
    b_dec = synth.normal_bf16("pin/sae_mm/bd", (d,), 0.1)
    tokens = [4, 0, 2]
    _, _, _, pre = oracle.sae_encode(h, tokens, W, b_enc, b_dec, 8, want_pre=True)
    U = bf16_vals(h[tokens]) - bf16_vals(b_dec)[None]
    ref = U @ bf16_vals(W).T + bf16_vals(b_enc)[None]
    assert np.allclose(pre, ref, rtol=0, atol=1e-12)


# ----------------------------------------------------------- clamp-decode

def test_clamp_equals_dense_recompute():
    d, m, k, T = 48, 96, 6, 5
    W_enc = synth.normal_bf16("pin/clamp/W", (m, d), 1 / np.sqrt(d))
    W_dec = synth.rownorm_bf16(W_enc)
    b_enc = synth.normal_bf16("pin/clamp/be", (m,), 0.1)
    b_dec = synth.normal_bf16("pin/clamp/bd", (d,), 0.1)
    h = synth.normal_bf16("pin/clamp/h", (T, d), 1.0)
    idx, val, _, _ = oracle.sae_encode(h, list(range(T)), W_enc, b_enc, b_dec, k)
    clamp_ids = np.array([int(idx[0, 0]), 5, 77, int(idx[2, 3])], np.int32)
    clamp_vals = np.array([10.0, 10.0, -2.5, 0.0], np.float32)
    tok_mask = np.array([1, 1, 1, 0, 1], np.uint32)
    out, delta = oracle.clamp_decode(h, tok_mask, 0, idx, val, W_dec, clamp_ids, clamp_vals,
                                     want_delta=True)
    Wd = bf16_vals(W_dec)
    for t in range(T):
        if not tok_mask[t]:
            assert np.array_equal(out[t], h[t])
            continue
        z = np.zeros(m)
        z[idx[t]] = bf16_vals(val[t])
        z2 = z.copy()
        z2[clamp_ids] = clamp_vals
        dense = z2 @ Wd - z @ Wd          # decode(z') - decode(z), all m latents
        assert np.allclose(delta[t], dense, rtol=0, atol=1e-12)


def test_clamp_to_current_value_is_identity():
    d, m, k = 32, 64, 4
    h = synth.normal_bf16("pin/clamp0/h", (2, d), 1.0)
    W_dec = synth.rownorm_bf16(synth.normal_bf16("pin/clamp0/W", (m, d), 1.0))
    idx = np.array([[3, 9, 1, 60], [2, 3, 4, 5]], np.int32)
    val = f32_to_bf16_torch(np.array([[2.5, 1.0, 0.5, 0.25], [4.0, 3.0, 2.0, 1.0]]))
    ids = np.array([9, 3], np.int32)
    # token 0 carries 9 -> 1.0, 3 -> 2.5; token 1 carries 3 -> 3.0 but not 9
    out, delta = oracle.clamp_decode(h, np.array([1, 0], np.uint32), 0, idx, val, W_dec, ids,
                                     np.array([1.0, 2.5], np.float32), want_delta=True)
    assert np.all(delta[0] == 0.0)
    assert np.array_equal(bf16_vals(out), bf16_vals(h))


def test_clamp_orthonormal_dictionary_moves_one_channel():
    d = m = 16
    W_dec = np.zeros((m, d), np.uint16)
    W_dec[np.arange(m), np.arange(d)] = 0x3F80
    h = f32_to_bf16_torch(np.arange(2 * d, dtype=np.float32).reshape(2, d) / 8)
    idx = np.array([[4, 7], [1, 2]], np.int32)
    val = f32_to_bf16_torch(np.array([[1.5, 0.5], [1.0, 1.0]]))
    out, delta = oracle.clamp_decode(h, np.array([1, 1], np.uint32), 0, idx, val, W_dec,
                                     np.array([7], np.int32), np.array([10.0], np.float32),
                                     want_delta=True)
    exp = np.zeros((2, d))
    exp[0, 7] = 10.0 - 0.5
    exp[1, 7] = 10.0
    assert np.array_equal(delta, exp)
    assert np.array_equal(out, f32_to_bf16_torch(bf16_vals(h) + exp))


# ----------------------------------------------------------------- ring

def brute_ring(rows, tok_mask, bit, req, layer, app, cap, row_bytes, head):
    slots = [None] * cap
    i = 0
    for t in range(len(tok_mask)):
        if (tok_mask[t] >> bit) & 1:
            hdr = np.array([t, req[t], layer, app], np.int32).view(np.uint8)
            slots[(head + i) % cap] = np.concatenate([hdr, rows[t]])
            i += 1
    return slots, head + i


@pytest.mark.parametrize("cap,head", [(8, 0), (8, 5), (3, 7), (64, 2 ** 40 + 3)])
def test_compact_brute_force(cap, head):
    rng = np.random.default_rng(cap + head % 97)
    T, pb = 20, 12
    rows = rng.integers(0, 256, (T, pb), dtype=np.uint8)
    tok_mask = rng.integers(0, 4, T).astype(np.uint32)
    req = rng.integers(0, 9, T).astype(np.int32)
    slots = np.full((cap, 16 + pb), 0xEE, np.uint8)
    seg_a, seg_b = rows[:, :8].copy(), rows[:, 8:].copy()
    out, new_head = oracle.compact([seg_a, seg_b], tok_mask, 1, req, 3, 11, slots, head)
    exp, exp_head = brute_ring(rows, tok_mask, 1, req, 3, 11, cap, 16 + pb, head)
    assert new_head == exp_head
    assert new_head - head == sum(int(m >> 1) & 1 for m in tok_mask)
    for s in range(cap):
        if exp[s] is None:
            assert np.all(out[s] == 0xEE)
        else:
            assert np.array_equal(out[s], exp[s])


# ---------------------------------------------------- conditional writes

def _gate_case(seed):
    rng = np.random.default_rng(seed)
    T, R, n_apps = 97, 9, 5
    req = rng.integers(-1, R, T).astype(np.int32)
    sub = rng.integers(0, 1 << n_apps, R).astype(np.uint32)
    return T, R, n_apps, req, sub, rng


@pytest.mark.parametrize("seed", range(4))
def test_route_gate_brute_force(seed):
    T, R, n_apps, req, sub, rng = _gate_case(seed)
    tm, cnt, lists, _ = oracle.route(req, T, sub, n_apps)
    sig = rng.normal(size=T).astype(np.float32)
    sig[rng.integers(0, T, 5)] = np.nan
    app, sbit, thr = 2, 4, 0.1
    tm2, cnt2, lists2 = oracle.route_gate(tm, cnt, lists, app, sig, thr, signal_bit=sbit)
    keep = [t for t in range(T) if (tm[t] >> app) & 1 and (tm[t] >> sbit) & 1 and sig[t] >= thr]
    assert cnt2[app] == len(keep) and list(lists2[app, :len(keep)]) == keep
    assert np.all(lists2[app, len(keep):] == -1)
    for t in range(T):
        assert ((tm2[t] >> app) & 1) == (t in keep)
        assert (tm2[t] & ~np.uint32(1 << app)) == (tm[t] & ~np.uint32(1 << app))
    others = [a for a in range(n_apps) if a != app]
    assert np.array_equal(lists2[others], lists[others]) and np.array_equal(cnt2[others], cnt[others])


def test_route_gate_per_request_and_limits():
    T, R, n_apps, req, sub, rng = _gate_case(11)
    tm, cnt, lists, _ = oracle.route(req, T, sub, n_apps)
    app = 1
    sig_r = rng.normal(size=R).astype(np.float32)
    tm2, cnt2, lists2 = oracle.route_gate(tm, cnt, lists, app, sig_r, 0.0, req=req)
    keep = [t for t in range(T) if (tm[t] >> app) & 1 and sig_r[req[t]] >= 0.0]
    assert list(lists2[app, :cnt2[app]]) == keep
    # -inf passes every finite signal, +inf none
    _, c_all, _ = oracle.route_gate(tm, cnt, lists, app, np.zeros(T, np.float32), -np.inf)
    _, c_none, _ = oracle.route_gate(tm, cnt, lists, app, np.zeros(T, np.float32), np.inf)
    assert c_all[app] == cnt[app] and c_none[app] == 0


@pytest.mark.parametrize("seed", range(3))
def test_route_trigger_brute_force(seed):
    T, R, n_apps, req, sub, rng = _gate_case(20 + seed)
    tm, cnt, lists, _ = oracle.route(req, T, sub, n_apps)
    V = 1000
    ids = rng.integers(-5, V + 5, T).astype(np.int32)
    trig = set(rng.choice(V, 60, replace=False).tolist())
    bits = np.zeros((V + 31) // 32, np.uint32)
    for v in trig:
        bits[v >> 5] |= np.uint32(1 << (v & 31))
    app = 3
    tm2, cnt2, lists2 = oracle.route_trigger(tm, cnt, lists, app, ids, bits, V)
    keep = [t for t in range(T) if (tm[t] >> app) & 1 and int(ids[t]) in trig]
    assert cnt2[app] == len(keep) and list(lists2[app, :len(keep)]) == keep
    assert all(((tm2[t] >> app) & 1) == (t in keep) for t in range(T))


# -------------------------------------------------------- router-logit write

def test_router_zero_offsets_is_identity():
    rng = np.random.default_rng(40)
    lg = f32_to_bf16_torch(rng.normal(0.0, 1.0, (9, 8)))
    out = oracle.router_write(lg, np.full(9, 0b11, np.uint32), [0, 1], np.zeros((2, 8), np.float32))
    assert np.array_equal(out, lg)


def test_router_minus_inf_removes_one_expert():
    """One app deactivates expert 5: only that entry of its tokens becomes
    -inf; the router's top-2 never picks it; unsubscribed rows keep their
    bits."""
    rng = np.random.default_rng(41)
    T, E = 16, 8
    lg = rng.normal(0.0, 1.0, (T, E)).astype(np.float32)
    lg[:, 5] += 10.0                                   # expert 5 would win everywhere
    off = np.zeros((1, E), np.float32)
    off[0, 5] = -np.inf
    tm = (np.arange(T) % 2).astype(np.uint32) << np.uint32(4)  # odd tokens carry bit 4
    out = oracle.router_write(lg, tm, [4], off)
    for t in range(T):
        if tm[t]:
            assert out[t, 5] == -np.inf
            keep = np.delete(np.arange(E), 5)
            assert np.array_equal(out[t, keep], lg[t, keep])
            assert 5 not in np.argsort(-out[t])[:2]
        else:
            assert np.array_equal(out[t], lg[t])
            assert np.argmax(out[t]) == 5


def test_router_sums_apps_in_order_and_rounds_once():
    """fp32 logits: the sum of the subscribed apps' offsets equals an exact
    math.fsum rounded once (the terms are chosen so that rounding after each
    addition would differ); app s is gated by bit app_bits[s]."""
    T, E = 4, 4
    lg = np.full((T, E), 1.0, np.float32)
    off = np.array([[2.0 ** -24, 0.0, 3.0, 0.0],
                    [2.0 ** -24, 0.0, -1.0, 0.0],
                    [0.0, 0.0, 0.5, 1e4]], np.float32)
    bits = [6, 2, 9]
    tm = np.array([(1 << 6) | (1 << 2), 1 << 9, (1 << 6) | (1 << 2) | (1 << 9), 1 << 3], np.uint32)
    out = oracle.router_write(lg, tm, bits, off)
    for t in range(T):
        sel = [s for s in range(3) if (tm[t] >> bits[s]) & 1]
        for e in range(E):
            exact = math.fsum([1.0] + [float(off[s, e]) for s in sel])
            assert out[t, e] == np.float32(exact)
    # 1 + 2^-24 + 2^-24 rounds once to 1 + 2^-23, not twice to 1
    assert out[0, 0] == np.float32(1.0 + 2.0 ** -23)
    assert np.array_equal(out[3], lg[3])               # bit 3 is no router app


def test_router_bf16_rounds_once_from_the_exact_sum():
    """bf16 logits: the result is the RNE of the exact fp64 sum (checked with
    the library fp32->bf16 cast on sums that are exact in fp32)."""
    rng = np.random.default_rng(42)
    T, E, n = 10, 8, 3
    lg = f32_to_bf16_torch(rng.integers(-64, 64, (T, E)) / 8.0)
    off = (rng.integers(-512, 512, (n, E)) / 256.0).astype(np.float32)
    tm = rng.integers(0, 8, T).astype(np.uint32)
    out = oracle.router_write(lg, tm, [0, 1, 2], off)
    lv = bf16_vals(lg)
    for t in range(T):
        if tm[t] == 0:
            assert np.array_equal(out[t], lg[t])
            continue
        acc = lv[t] + sum(off[s].astype(np.float64) for s in range(n) if (tm[t] >> s) & 1)
        assert np.array_equal(acc.astype(np.float32).astype(np.float64), acc)
        assert np.array_equal(out[t], f32_to_bf16_torch(acc))
