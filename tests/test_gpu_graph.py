"""HIP-graph capture of a whole hook step: one capture, replays with new
device-side subscriptions and alpha, each replay checked against the eager
run and the oracle; replays of the same inputs are bit-identical (no float
atomics anywhere in the step)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_steer, check_topk, torch_bits

pytestmark = pytest.mark.gpu


def _mixed_workload():
    # decode batch with steering, probes and an SAE with a ring
    wl = synth.make("c2", d=512, T=200, n_layers=2)
    sae_wl = synth.make("c3", d=512, m=1024, k=16, T=200, ring_capacity=128)
    s = sae_wl.layers[0].saes[0]
    s.bit = 8
    wl.n_apps = 9
    wl.sub = wl.sub | (sae_wl.sub << np.uint32(8))
    wl.layers[1].saes.append(s)
    return wl


def _snapshot(step):
    out = {}
    for li, lay in enumerate(step.layers):
        out[f"h{li}"] = torch_bits(lay.h).copy()
        for pi, p in enumerate(lay.probes):
            out[f"p{li}.{pi}"] = p.logit.cpu().numpy().copy()
        for si, s in enumerate(lay.saes):
            out[f"i{li}.{si}"] = s.idx.cpu().numpy().copy()
            out[f"v{li}.{si}"] = torch_bits(s.val).copy()
    return out


def test_graph_replay_matches_eager_and_is_deterministic():
    from paper_2607_22595_amd.hookstep import HookStep
    wl = _mixed_workload()
    step = HookStep(wl)
    step.reset()
    step.run()
    torch.cuda.synchronize()
    eager = _snapshot(step)

    g = torch.cuda.CUDAGraph()
    step.reset()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step.run()
    for rep in range(3):
        step.reset()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = _snapshot(step)
        for key in eager:
            assert np.array_equal(snap[key], eager[key]), (rep, key)
    ring = step.layers[1].saes[0].ring
    n_sub = int(np.count_nonzero((wl.sub >> np.uint32(8)) & 1))
    assert int(ring.head[0].item()) == 4 * n_sub      # eager + 3 replays

    # new subscriptions and alpha, written into the same device buffers
    rng = np.random.default_rng(5)
    new_sub = rng.integers(0, 2 ** 9, wl.R_max).astype(np.uint32)
    new_alpha = rng.uniform(-8, 8, wl.alpha.shape).astype(np.float32)
    step.sub.copy_(torch.from_numpy(new_sub.view(np.int32)))
    step.alpha.copy_(torch.from_numpy(new_alpha))
    step.reset()
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    tm, cnt, lists, err = oracle.route(wl.req, wl.T_valid, new_sub, wl.n_apps)
    assert np.array_equal(step.route.tok_mask.cpu().numpy().view(np.uint32), tm)
    for L, lay in zip(wl.layers, step.layers):
        bits = [s.bit for s in L.steer]
        ref = oracle.steer(L.h, tm, wl.req, np.stack([s.v for s in L.steer]), bits, new_alpha)
        rows = (tm & np.uint32(sum(1 << b for b in bits))) != 0
        check_steer(torch_bits(lay.h), ref, L.h, rows)
    s, sd = wl.layers[1].saes[0], step.layers[1].saes[0]
    toks = lists[8, :cnt[8]]
    idx_ref, _, _, pre = oracle.sae_encode(wl.layers[1].h, toks, s.W_enc, s.b_enc, s.b_dec, s.k,
                                           want_pre=True)
    idx = sd.idx.cpu().numpy()
    val = torch_bits(sd.val)
    for q, t in enumerate(toks):
        check_topk(idx[t], val[t], idx_ref[q], pre[q], s.k)


def test_all_zero_mask_step_writes_nothing():
    """'Don't use, don't pay': with no subscriptions nothing but the routing
    table is written."""
    from paper_2607_22595_amd.hookstep import HookStep
    wl = _mixed_workload()
    wl.sub[:] = 0
    step = HookStep(wl)
    for lay in step.layers:
        for p in lay.probes:
            p.logit.fill_(float("nan"))
        for s in lay.saes:
            s.idx.fill_(-3)
    step.run()
    torch.cuda.synchronize()
    for L, lay in zip(wl.layers, step.layers):
        assert np.array_equal(torch_bits(lay.h), L.h)
        for p in lay.probes:
            assert torch.isnan(p.logit).all()
        for s in lay.saes:
            assert (s.idx == -3).all()
            assert int(s.ring.head[0].item()) == 0
