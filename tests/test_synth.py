"""The seeded input generator: determinism, distributions, workload recipes."""
import numpy as np
import torch

import synth


def test_streams_are_deterministic_and_independent():
    a = synth.normal_bf16("t/x", (1000,), 1.0)
    b = synth.normal_bf16("t/x", (1000,), 1.0)
    c = synth.normal_bf16("t/y", (1000,), 1.0)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)
    # a prefix of a longer draw is the shorter draw (counter-based streams)
    long = synth.normal_bf16("t/x", (5000,), 1.0)
    assert np.array_equal(long[:1000], a)
    # a different seed gives a different stream
    assert not np.array_equal(synth.normal_bf16("t/x", (1000,), 1.0, seed=1), a)


def test_normal_moments():
    x = synth.normal_f32("t/moments", (400000,), 2.0, mean=0.5).astype(np.float64)
    # sample mean and variance of 4e5 draws: 5-sigma bounds
    assert abs(x.mean() - 0.5) < 5 * 2.0 / np.sqrt(x.size)
    assert abs(x.var() - 4.0) < 5 * 4.0 * np.sqrt(2.0 / x.size)
    # standardised third and fourth moments of a normal: 0 and 3
    z = (x - x.mean()) / x.std()
    assert abs((z ** 3).mean()) < 0.02
    assert abs((z ** 4).mean() - 3.0) < 0.05


def test_generator_bf16_rounding_matches_torch():
    # For values exactly representable in fp32, torch's fp32 -> bf16
    # conversion is round-to-nearest-even: an independent implementation.
    rng = np.random.default_rng(1)
    vals = np.concatenate([rng.standard_normal(2000).astype(np.float32),
                           (rng.standard_normal(2000) * 1e-30).astype(np.float32),
                           np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 2 ** -133,
                                     3e38, 0.0], np.float32)])
    ref = torch.from_numpy(vals).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([synth.bf16_from_double(float(v)) for v in vals], np.uint16)
    assert np.array_equal(got, ref)


def test_permutation_is_a_permutation():
    p = synth.permutation("t/perm", 1000)
    assert sorted(p.tolist()) == list(range(1000))
    assert not np.array_equal(p, np.arange(1000))


def test_rownorm_unit_rows():
    W = synth.normal_bf16("t/W", (64, 256), 1 / 16)
    D = synth.bf16_bits_to_f32(synth.rownorm_bf16(W)).astype(np.float64)
    norms = np.linalg.norm(D, axis=1)
    assert np.all(np.abs(norms - 1.0) < 256 ** 0.5 * 2 ** -8)


def test_c1_recipe():
    wl = synth.make("c1")
    assert wl.dtype == "f32" and wl.d == 256 and wl.T_max == 16 and wl.R_max == 4
    assert set(wl.req.tolist()) <= {0, 1, 2, 3}
    assert wl.sub.tolist() == [1, 2, 3, 2]
    assert np.all(wl.alpha == 4.0)


def test_c3_recipe_small():
    wl = synth.make("c3", d=256, m=1024, k=16, T=64)
    assert int(np.count_nonzero(wl.sub)) == 32
    sae = wl.layers[0].saes[0]
    assert sae.W_enc.shape == (1024, 256) and sae.ring_capacity == 256


def test_c4_ragged_layout():
    wl = synth.make("c4", d=64, m=256, k=8)
    cu = wl.cu_seqlens
    lens = np.diff(cu)
    assert cu[0] == 0 and cu[-1] == 8192 and lens.size == 16
    assert lens.min() >= 128 and lens.max() <= 1024
    assert np.array_equal(wl.req, np.repeat(np.arange(16), lens))


def test_c5_recipe_small():
    wl = synth.make("c5", d=128, T=32, m=512, k=8)
    assert wl.n_apps == 32
    L = wl.layers[0]
    assert len(L.steer) == 16 and len(L.probes) == 8 and len(L.saes) == 8
    for s in L.saes:
        assert s.clamp_ids.size == 4 and len(set(s.clamp_ids.tolist())) == 4
        assert np.all(s.clamp_vals == 10.0)
        assert s.W_dec.shape == s.W_enc.shape
