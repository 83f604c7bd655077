"""xmix_sae_encode_topk_noalloc (the encode without a workspace argument,
whose scratch is the library's static per-GPU array) against
xmix_sae_encode_topk with a caller workspace: the same kernels, so the same
bits, on two calls in a row, the second smaller than the first (the array
keeps the first call's contents), and against the oracle on sampled tokens."""
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


def _dev_bits(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)


def _dev_i32(a):
    a = np.ascontiguousarray(a)
    return torch.from_numpy(a.view(np.int32) if a.dtype == np.uint32 else a.astype(np.int32)).cuda()


def _both(px, wl, fold):
    sae = wl.layers[0].saes[0]
    rt = px.Route(wl.T_max, wl.n_apps)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    px.xmix_route_build(_dev_i32(wl.req), torch.tensor([wl.T_valid], dtype=torch.int32,
                                                       device="cuda"),
                        _dev_i32(wl.sub), rt, err)
    h = _dev_bits(wl.layers[0].h)
    W = px.xmix_sae_pack_encoder(_dev_bits(sae.W_enc))
    be, bd = _dev_bits(sae.b_enc), _dev_bits(sae.b_dec)
    c = None
    if fold:
        c = torch.empty(sae.m, dtype=torch.float32, device="cuda")
        px.xmix_sae_fold_bias(W, be, bd, c)
    out = []
    for noalloc in (False, True):
        idx = torch.full((wl.T_max, sae.k), -7, dtype=torch.int32, device="cuda")
        val = torch.zeros((wl.T_max, sae.k), dtype=torch.bfloat16, device="cuda")
        if noalloc:
            px.xmix_sae_encode_topk_noalloc(h, rt, sae.bit, W, be, bd, c, sae.k, idx, val)
        else:
            ws = torch.empty(px.sae_encode_workspace(wl.T_max, wl.d, sae.m, sae.k),
                             dtype=torch.uint8, device="cuda")
            px.xmix_sae_encode_topk(h, rt, sae.bit, W, be, bd, c, sae.k, idx, val, ws)
        torch.cuda.synchronize()
        out.append((idx.cpu().numpy(), torch_bits(val)))
    (ia, va), (ib, vb) = out
    assert np.array_equal(ia, ib) and np.array_equal(va, vb)
    toks = rt.app_tokens[sae.bit, :int(rt.app_count[sae.bit].item())].cpu().numpy()
    assert len(toks) > 0
    unsub = np.setdiff1d(np.arange(wl.T_max), toks)
    assert np.all(ib[unsub] == -7)                 # rows of unsubscribed tokens untouched
    sample = toks[:: max(1, len(toks) // 12)]
    idx_ref, _, _, pre = oracle.sae_encode(wl.layers[0].h, sample, sae.W_enc, sae.b_enc,
                                           sae.b_dec, sae.k, want_pre=True)
    for q, t in enumerate(sample):
        check_topk(ib[t], vb[t], idx_ref[q], pre[q], sae.k)


def test_noalloc_encode_matches_workspace_encode_twice(px):
    # first: the decode SAE shape (d=4096, m=65536, k=64, 256 slots, 128
    # subscribed); second: a smaller batch, dictionary and k, no folded bias
    # (the fold goes to the static array too)
    _both(px, synth.make("c3"), fold=True)
    _both(px, synth.make("c3", d=512, m=2048, k=16, T=70, n_sub=40, seed=3), fold=False)


def test_noalloc_encode_refuses_more_than_the_static_array(px):
    wl = synth.make("c3", d=256, m=65536, k=64, T=1024, n_sub=8, seed=5)
    sae = wl.layers[0].saes[0]
    need = px.sae_encode_workspace(wl.T_max, wl.d, sae.m, sae.k)
    assert need > px.XMIX_STATIC_SCRATCH_BYTES
    rt = px.Route(wl.T_max, wl.n_apps)
    W = px.xmix_sae_pack_encoder(_dev_bits(sae.W_enc))
    idx = torch.full((wl.T_max, sae.k), -7, dtype=torch.int32, device="cuda")
    val = torch.zeros((wl.T_max, sae.k), dtype=torch.bfloat16, device="cuda")
    h = _dev_bits(wl.layers[0].h)
    with pytest.raises(px.XmixError) as e:
        px.xmix_sae_encode_topk_noalloc(h, rt, 0, W, _dev_bits(sae.b_enc), _dev_bits(sae.b_dec),
                                        None, sae.k, idx, val)
    assert e.value.status == px.XMIX_E_UNSUPPORTED
    torch.cuda.synchronize()
    assert np.all(idx.cpu().numpy() == -7)
