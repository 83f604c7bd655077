"""The library's own step graph (xmix_graph_*): a multi-layer hook step
captured once on a stream, replayed with per-step values changed in device
memory, and with whole parameter buffers swapped through kernel-node
parameter updates (redirect).  Every replay is compared with an eager run
of the same inputs (bit-identical: the same kernels on the same data), and
the redirected steering against the oracle."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import check_steer, torch_bits

pytestmark = pytest.mark.gpu


def _workload():
    # 4 hooked layers: bits 0-3 steer, 4-7 probe, plus a clamp SAE on layer 2
    wl = synth.make("c2", d=512, T=160, n_layers=4)
    c5 = synth.make("c5", d=512, T=160, m=1024, k=16, n_steer=0, n_probe=0, n_clamp_apps=1)
    s = c5.layers[0].saes[0]
    s.bit = 8
    wl.n_apps = 9
    wl.sub = wl.sub | (c5.sub << np.uint32(8))
    wl.layers[2].saes.append(s)
    return wl


def _h(step):
    return [torch_bits(lay.h).copy() for lay in step.layers]


def _eager(step):
    step.reset()
    step.run()
    torch.cuda.synchronize()
    return _h(step)


def _replay(step, g):
    step.reset()
    torch.cuda.synchronize()
    g.launch()
    g.stream.synchronize()
    return _h(step)


@pytest.fixture(scope="module")
def captured():
    import paper_2607_22595_amd as px
    from paper_2607_22595_amd.hookstep import HookStep
    wl = _workload()
    step = HookStep(wl)
    step.run()
    torch.cuda.synchronize()
    stream = torch.cuda.Stream()
    g = px.Graph(lambda: step.run(stream), stream)
    yield wl, step, g
    torch.cuda.synchronize()
    g.close()


def test_step_graph_replays_match_eager(captured):
    wl, step, g = captured
    # 4 x (probes and steering in one pass; the first also builds the
    # routing), encode (candidates + merge) and clamp
    assert g.kernel_nodes >= 7
    ref = _eager(step)
    for _ in range(3):
        got = _replay(step, g)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b)


def test_in_memory_values_change_without_update(captured):
    """New alpha, subscriptions and clamp values written into the device
    buffers the graph reads: the next replay uses them, no update needed."""
    wl, step, g = captured
    rng = np.random.default_rng(3)
    s = step.layers[2].saes[0]
    for rep in range(2):
        step.alpha.copy_(torch.from_numpy(rng.uniform(-8, 8, tuple(step.alpha.shape))
                                          .astype(np.float32)))
        step.sub.copy_(torch.from_numpy(rng.integers(0, 1 << 9, step.sub.numel())
                                        .astype(np.uint32).view(np.int32)))
        s.clamp_vals.copy_(torch.from_numpy(rng.uniform(-5, 15, s.clamp_vals.numel())
                                            .astype(np.float32)))
        torch.cuda.synchronize()
        got = _replay(step, g)
        ref = _eager(step)
        for a, b in zip(got, ref):
            assert np.array_equal(a, b), f"replay {rep}"


def test_redirect_steering_alpha_by_node_update(captured):
    """Swap the whole alpha buffer by a kernel-node update: one argument per
    steering node (4 layers) changes; the replay equals an eager run with the
    new buffer and, on layer 0, the oracle's steering."""
    wl, step, g = captured
    alpha0 = step.alpha
    rng = np.random.default_rng(4)
    alpha1 = torch.from_numpy(rng.uniform(-8, 8, tuple(alpha0.shape)).astype(np.float32)).cuda()
    n = g.redirect(alpha0, alpha1)
    assert n == 4
    got = _replay(step, g)
    step.alpha = alpha1                      # the eager run reads the new buffer too
    try:
        ref = _eager(step)
    finally:
        step.alpha = alpha0
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)
    # layer 0 against the oracle: its probes only read, so h0 is the steered input
    lay0, L0 = step.layers[0], wl.layers[0]
    tm, _, _, _ = oracle.route(wl.req, wl.T_valid, torch_sub(step), wl.n_apps)
    v = np.stack([a.v for a in L0.steer])
    h_ref = oracle.steer(L0.h, tm, wl.req, v, [a.bit for a in L0.steer], alpha1.cpu().numpy())
    check_steer(got[0], h_ref, L0.h, (tm & 0xF) != 0)
    assert g.redirect(alpha1, alpha0) == 4   # and back
    got = _replay(step, g)
    ref = _eager(step)
    for a, b in zip(got, ref):
        assert np.array_equal(a, b)


def torch_sub(step):
    return step.sub.cpu().numpy().view(np.uint32)


def test_redirect_subscriptions_and_unknown_buffer(captured):
    wl, step, g = captured
    sub0 = step.sub
    sub1 = torch.zeros_like(sub0)            # nobody subscribed
    assert g.redirect(sub0, sub1) == 1       # the route build reads it once
    got = _replay(step, g)
    for lay, a in zip(step.layers, got):
        assert np.array_equal(a, torch_bits(lay.h_in))
    assert g.redirect(sub1, sub0) == 1
    other = torch.zeros(16, dtype=torch.float32, device="cuda")
    assert g.redirect(other, torch.zeros_like(other)) == 0


def test_capture_after_dropping_a_torch_graph_in_a_cycle(captured):
    """A torch CUDA graph left in a reference cycle is collected before the
    library's capture starts, not during it (collected during the capture,
    its teardown would make a HIP call that capture forbids)."""
    import gc
    import paper_2607_22595_amd as px
    wl, step, _ = captured
    x = torch.zeros(1024, device="cuda")
    tg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(tg):
        x.add_(1.0)
    holder = {"graph": tg}
    holder["self"] = holder  # a cycle: only the collector frees it
    del tg, holder
    stream = torch.cuda.Stream()
    g = px.Graph(lambda: step.run(stream), stream)
    try:
        assert gc.isenabled()
        ref = _eager(step)
        assert all(np.array_equal(a, b) for a, b in zip(_replay(step, g), ref))
    finally:
        torch.cuda.synchronize()
        g.close()


def test_decode_sae_step_graph_with_routing_in_the_encode():
    """A decode SAE step whose routing is built inside the encode launch:
    the captured step replays like the eager one, and redirecting the
    subscription buffer reaches the encode kernel (no token encoded, the
    ring head unchanged), and back."""
    import paper_2607_22595_amd as px
    from paper_2607_22595_amd.hookstep import HookStep
    wl = synth.make("c3", d=512, m=2048, k=16, T=200, ring_capacity=256)
    step = HookStep(wl)
    s = step.layers[0].saes[0]
    step.run()
    torch.cuda.synchronize()
    n = int(step.route.app_count[0].item())
    toks = step.route.app_tokens[0, :n].long()
    assert n > 0
    idx_ref, val_ref = s.idx[toks].clone(), s.val[toks].clone()
    stream = torch.cuda.Stream()
    g = px.Graph(lambda: step.run(stream), stream)

    def replay():
        s.idx.fill_(-3)
        torch.cuda.synchronize()
        g.launch()
        g.stream.synchronize()

    try:
        assert g.kernel_nodes == 2  # the encode (with the routing) and the merge
        replay()
        assert torch.equal(s.idx[toks], idx_ref) and torch.equal(s.val[toks], val_ref)
        head = int(s.ring.head[0].item())
        sub1 = torch.zeros_like(step.sub)
        assert g.redirect(step.sub, sub1) == 1   # read once, by the encode
        replay()
        assert bool((s.idx == -3).all()) and int(s.ring.head[0].item()) == head
        assert int(step.route.app_count[0].item()) == 0
        assert g.redirect(sub1, step.sub) == 1
        replay()
        assert torch.equal(s.idx[toks], idx_ref)
    finally:
        torch.cuda.synchronize()
        g.close()


def test_redirect_reaches_buffers_inside_batched_calls():
    """A layer with three clamp SAEs runs as one batched encode and one
    batched clamp, whose app descriptors hold the buffers: redirecting one
    app's clamp values changes one argument (the batched clamp), and one
    app's dictionary two (the batched encode and merge); each replay equals
    an eager run with the new buffer, and the graph goes back."""
    import paper_2607_22595_amd as px
    from paper_2607_22595_amd.hookstep import HookStep
    wl = synth.make("c5", d=512, T=160, m=1024, k=16, n_steer=2, n_probe=1, n_clamp_apps=3,
                    seed=21)
    step = HookStep(wl)
    saes = step.layers[0].saes

    def snap():
        torch.cuda.synchronize()
        return [torch_bits(step.layers[0].h).copy()] + \
            [x for s in saes for x in (s.idx.cpu().numpy(), torch_bits(s.val))]

    def eager():
        step.reset()
        step.run()
        return snap()

    def same(a, b):
        return all(np.array_equal(x, y) for x, y in zip(a, b))

    ref0 = eager()
    stream = torch.cuda.Stream()
    g = px.Graph(lambda: step.run(stream), stream)

    def replay():
        step.reset()
        torch.cuda.synchronize()
        g.launch()
        g.stream.synchronize()
        return snap()

    try:
        assert same(replay(), ref0)
        s1 = saes[1]
        vals0 = s1.clamp_vals
        vals1 = (vals0 * -1.5 + 3.0).contiguous()
        assert g.redirect(vals0, vals1) == 1
        got = replay()
        s1.clamp_vals = vals1
        try:
            ref = eager()
        finally:
            s1.clamp_vals = vals0
        assert same(got, ref) and not same(got, ref0)
        assert g.redirect(vals1, vals0) == 1
        # app 2's dictionary swapped for a copy of app 0's (same shape)
        s2 = saes[2]
        W0 = s2.W_enc
        W1 = saes[0].W_enc.clone()
        assert g.redirect(W0.packed, W1.packed) == 2
        got = replay()
        s2.W_enc = W1
        try:
            ref = eager()
        finally:
            s2.W_enc = W0
        assert same(got, ref) and not same(got, ref0)
        assert g.redirect(W1.packed, W0.packed) == 2
        assert same(replay(), ref0)
    finally:
        torch.cuda.synchronize()
        g.close()
