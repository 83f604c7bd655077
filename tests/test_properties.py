"""Property tests (hypothesis, small shapes): routing invariants of the
oracle on the CPU, and GPU routing, steering and readback against the
oracle on generated batches (padding, bad ids, ragged T_valid, any mask)."""
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
