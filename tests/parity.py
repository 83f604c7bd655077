"""Comparison rules of the GPU path against the CPU oracle.

Tolerances (floating point) and exactness (integer, index and byte work):
  - routing, ring compaction: bit-exact;
  - steering: within 1 bf16 ulp of the oracle value, ulp(x) = 2^(floor(log2|x|) - 7);
    unsubscribed rows bit-identical;
  - probe scores: 1e-3 relative; logits: 1e-3 relative with an absolute
    floor of 1e-3 * sum_i |w_i h_i|;
  - SAE top-k: |S| = k without duplicates; every index in the symmetric
    difference of the GPU and oracle sets lies within 1e-3 relative of the
    oracle's k-th pre-activation; values of common indices within 2e-2
    relative (absolute floor of one bf16 ulp of the k-th value for values
    that round to tiny numbers);
  - decoded delta: ||delta_gpu - delta_or||_2 <= 2e-2 ||delta_or||_2;
    residual: |h'_gpu - h'_or| <= ulp(h'_or) + 2e-2 ||delta_or||_inf.
"""
import numpy as np

import synth


def bf16_f64(bits):
    return synth.bf16_bits_to_f32(np.asarray(bits).view(np.uint16)).astype(np.float64)


def bf16_ulp(x):
    """ulp(x) = 2^(floor(log2|x|) - 7); the smallest normal's ulp at 0."""
    ax = np.abs(np.asarray(x, np.float64))
    ax = np.maximum(ax, 2.0 ** -126)
    return np.exp2(np.floor(np.log2(ax)) - 7)


def torch_bits(t):
    """A GPU bf16 tensor -> numpy uint16 bit patterns."""
    import torch
    return t.detach().cpu().view(torch.int16).numpy().view(np.uint16)


def check_steer(h_gpu_bits, h_ref_bits, h_in_bits, steered_rows, is_bf16=True):
    """Returns the max error in ulps over steered rows; asserts the rule."""
    if is_bf16:
        g = bf16_f64(h_gpu_bits)
        r = bf16_f64(h_ref_bits)
    else:
        g = np.asarray(h_gpu_bits, np.float64)
        r = np.asarray(h_ref_bits, np.float64)
    rows = np.asarray(steered_rows, bool)
    untouched = ~rows
    assert np.array_equal(np.asarray(h_gpu_bits)[untouched], np.asarray(h_in_bits)[untouched]), \
        "unsubscribed rows changed"
    if not rows.any():
        return 0.0
    err = np.abs(g[rows] - r[rows]) / bf16_ulp(r[rows])
    worst = float(err.max())
    assert worst <= 1.0, f"steering error {worst} ulp"
    return worst


def check_probe(logit_gpu, score_gpu, logit_ref, score_ref, mask, abs_floor):
    m = np.asarray(mask, bool)
    if not m.any():
        return
    sg, sr = score_gpu[m], score_ref[m]
    assert np.all(np.abs(sg - sr) <= 1e-3 * np.abs(sr)), \
        f"score rel err {np.max(np.abs(sg - sr) / np.abs(sr))}"
    lg, lr = logit_gpu[m], logit_ref[m]
    tol = np.maximum(1e-3 * np.abs(lr), 1e-3 * abs_floor[m])
    assert np.all(np.abs(lg - lr) <= tol), f"logit err {np.max(np.abs(lg - lr) - tol)}"


def check_topk(idx_gpu, val_gpu_bits, idx_ref, pre_ref, k):
    """One token.  idx_gpu/val_gpu_bits: GPU row; idx_ref: oracle row;
    pre_ref: the oracle's full pre-activation vector (fp64).
    Returns the number of boundary swaps."""
    ig = np.asarray(idx_gpu, np.int64)
    assert ig.size == k and len(set(ig.tolist())) == k, "duplicate or missing indices"
    assert np.all((ig >= 0) & (ig < pre_ref.size)), "index out of range"
    kth = np.sort(pre_ref)[::-1][k - 1]
    diff = set(ig.tolist()) ^ set(np.asarray(idx_ref).tolist())
    for j in diff:
        assert abs(pre_ref[j] - kth) <= 1e-3 * abs(kth), \
            f"index {j} (pre {pre_ref[j]}) outside the tie band of the k-th value {kth}"
    vg = bf16_f64(val_gpu_bits)
    exact = np.maximum(pre_ref[ig], 0.0)
    tol = np.maximum(2e-2 * exact, bf16_ulp(max(abs(kth), 1e-30)))
    assert np.all(np.abs(vg - exact) <= tol), f"value err {np.max(np.abs(vg - exact) - tol)}"
    # output order: value non-increasing
    assert np.all(np.diff(vg) <= 0), "values not in descending order"
    return len(diff) // 2


def check_delta(delta_gpu, delta_ref):
    n = np.linalg.norm(delta_ref)
    assert np.linalg.norm(delta_gpu - delta_ref) <= 2e-2 * n + 1e-30


def check_residual(h_gpu_bits, h_ref_bits, delta_ref):
    g, r = bf16_f64(h_gpu_bits), bf16_f64(h_ref_bits)
    tol = bf16_ulp(r) + 2e-2 * np.max(np.abs(delta_ref))
    assert np.all(np.abs(g - r) <= tol)
