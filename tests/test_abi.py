"""The C-ABI library loads and exports every entry point its header declares.

Runs without a GPU: only host-side calls are made (argument checks that
return before any launch, and workspace-size queries)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "xmix.h")
LIB = os.path.join(ROOT, "paper_2607_22595_amd", "libxmix.so")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(xmix_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    return ctypes.CDLL(LIB)


def test_header_declares_the_six_hot_path_calls():
    fns = declared_functions()
    for name in ("xmix_route_build", "xmix_steer_apply", "xmix_probe_score",
                 "xmix_sae_encode_topk", "xmix_sae_clamp_decode", "xmix_readback_compact"):
        assert name in fns


def test_every_declared_symbol_is_exported(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT\s+(xmix_\w+)", out))
    missing = [f for f in declared_functions() if f not in exported]
    assert not missing, missing
    for f in declared_functions():
        assert hasattr(lib, f)


def test_binding_wraps_every_symbol():
    import paper_2607_22595_amd as px
    assert sorted(px.EXPORTED) == declared_functions()


def test_host_validation_rejects_before_launch(lib):
    lib.xmix_route_build.restype = ctypes.c_int
    lib.xmix_steer_apply.restype = ctypes.c_int
    lib.xmix_sae_encode_topk.restype = ctypes.c_int
    lib.xmix_readback_compact.restype = ctypes.c_int
    lib.xmix_status_string.restype = ctypes.c_char_p
    # null pointers and missing route -> XMIX_E_INVAL (1), nothing launched
    assert lib.xmix_route_build(None, None, None, 1, None, None, None) == 1
    assert lib.xmix_steer_apply(None, 1, 64, None, None, None, None, None, 1, 1, None) == 1
    assert lib.xmix_sae_encode_topk(None, 64, None, 0, None, None, None, None, 8,
                                    None, None, None, ctypes.c_size_t(0), None) == 1
    assert lib.xmix_readback_compact(None, None, 1, None, 0, None, 0, 0, None, None) == 1
    lib.xmix_router_write.restype = ctypes.c_int
    assert lib.xmix_router_write(None, 0, 8, None, None, None, 1, None) == 1
    lib.xmix_route_sae_encode_candidates.restype = ctypes.c_int
    assert lib.xmix_route_sae_encode_candidates(None, None, None, 1, None, None, None, 256, 0,
                                                None, None, None, None, 8, None,
                                                ctypes.c_size_t(0), None) == 1
    lib.xmix_steer_probe.restype = ctypes.c_int
    assert lib.xmix_steer_probe(None, 1, 64, None, None, None, None, None, 1, 1, None, None,
                                None, 1, None, None, None) == 1
    assert lib.xmix_status_string(3) == b"workspace missing or too small"


def test_workspace_queries(lib):
    lib.xmix_sae_encode_workspace.restype = ctypes.c_size_t
    lib.xmix_probe_workspace.restype = ctypes.c_size_t
    # decode SAE: 256 token slots, m = 65536 (256 slices), k = 64: the
    # folded bias, then per (token, slice) a block of `cap` candidate pairs
    # (8 bytes each) plus a count and a threshold, 8 <= cap <= 64
    fold = 65536 * 4
    ws = lib.xmix_sae_encode_workspace(256, 4096, 65536, 64)
    per_slot, rem = divmod(ws - fold, 256 * 256)
    assert rem == 0 and (per_slot - 8) % 8 == 0
    assert 8 <= (per_slot - 8) // 8 <= 64
    assert lib.xmix_probe_workspace(8192, 4, 1) == 8192 * 4 * 4
    assert lib.xmix_probe_workspace(8192, 4, 0) == 0


def test_encode_rejects_unsupported_shapes_on_the_host(lib):
    """Fake (never dereferenced) device addresses: every case below is
    refused by the host-side checks before anything is launched."""
    import paper_2607_22595_amd as px
    f = lib.xmix_sae_encode_topk
    f.restype = ctypes.c_int
    f.argtypes = None
    rt = px.XmixRoute(0x10000, 0x20000, 0x30000, 256, 1)
    A = 0x100000   # 16-byte aligned fake address

    def call(d=4096, m=65536, k=64, ws_bytes=1 << 40, app_bit=0, c_fold=A, dict_d=None,
             layout=px.XMIX_SAE_DICT_TILED):
        w = px.XmixSaeDict(A, m, d if dict_d is None else dict_d, layout)
        return f(ctypes.c_void_p(A), d, ctypes.byref(rt), app_bit, ctypes.byref(w),
                 ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_void_p(c_fold), k,
                 ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_void_p(A),
                 ctypes.c_size_t(ws_bytes), None)
    assert call(d=320) == 1            # d must be a multiple of 256
    assert call(m=300) == 1            # m must be a multiple of 256
    assert call(k=65) == 1             # k <= 64
    assert call(k=0) == 1
    assert call(app_bit=1) == 1        # bit outside the route's apps
    assert call(m=262144, k=64) == 2   # too many merge candidates per token
    assert call(ws_bytes=1024) == 3    # workspace too small


def test_dictionary_must_come_from_the_packer(lib):
    """A row-major matrix cannot reach the encode in place of the packed
    dictionary: the calls take a descriptor that only xmix_sae_pack_encoder
    fills, and refuse one without its layout tag or of another width."""
    import paper_2607_22595_amd as px
    A = 0x100000
    rt = px.XmixRoute(0x10000, 0x20000, 0x30000, 256, 1)
    enc = lib.xmix_sae_encode_topk
    enc.restype = ctypes.c_int
    enc.argtypes = None
    fold = lib.xmix_sae_fold_bias
    fold.restype = ctypes.c_int
    fold.argtypes = None

    def call(w):
        return enc(ctypes.c_void_p(A), 4096, ctypes.byref(rt), 0,
                   None if w is None else ctypes.byref(w), ctypes.c_void_p(A),
                   ctypes.c_void_p(A), ctypes.c_void_p(A), 64, ctypes.c_void_p(A),
                   ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_size_t(1 << 40), None)
    # a descriptor filled by hand around a row-major matrix has no layout tag
    assert call(px.XmixSaeDict(A, 65536, 4096, 0)) == 1
    assert call(px.XmixSaeDict(A, 65536, 4096, px.XMIX_SAE_DICT_TILED ^ 1)) == 1
    assert call(px.XmixSaeDict(A, 65536, 2048, px.XMIX_SAE_DICT_TILED)) == 1  # width
    assert call(px.XmixSaeDict(0, 65536, 4096, px.XMIX_SAE_DICT_TILED)) == 1  # no pieces
    assert call(None) == 1
    assert fold(ctypes.byref(px.XmixSaeDict(A, 65536, 4096, 0)), ctypes.c_void_p(A),
                ctypes.c_void_p(A), ctypes.c_void_p(A), None) == 1
    # the binding refuses anything but a packed dictionary object
    with pytest.raises(TypeError):
        px._dict(object())
    # the C prototypes take the descriptor, not a bare pointer
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for fn in ("xmix_sae_encode_topk", "xmix_sae_encode_candidates", "xmix_sae_merge_topk",
               "xmix_route_sae_encode_candidates", "xmix_sae_encode_topk_ring",
               "xmix_sae_merge_topk_ring", "xmix_sae_fold_bias"):
        proto = re.search(fn + r"\s*\(([^;]*)\)\s*;", text).group(1)
        assert "const xmix_sae_dict *dict" in proto and "W_packed" not in proto, fn


CEIL_HEADER = os.path.join(ROOT, "include", "xmix_ceiling.h")
CEIL_LIB = os.path.join(ROOT, "paper_2607_22595_amd", "libxmix_ceiling.so")


def test_ceiling_library_exports_its_header():
    """The measured-ceiling aid (a benchmark tool beside the hook step)."""
    if not os.path.exists(CEIL_LIB):
        import __graft_entry__
        __graft_entry__.build()
    text = re.sub(r"/\*.*?\*/", "", open(CEIL_HEADER).read(), flags=re.S)
    declared = sorted(set(re.findall(r"\b(xmix_[a-z_0-9]+)\s*\(", text)))
    assert declared == ["xmix_ceiling_mfma", "xmix_ceiling_read"]
    out = subprocess.run(["nm", "-D", "--defined-only", CEIL_LIB], capture_output=True,
                         text=True, check=True).stdout
    assert sorted(set(re.findall(r"\bT\s+(xmix_\w+)", out))) == declared
    lib = ctypes.CDLL(CEIL_LIB)
    lib.xmix_ceiling_read.restype = ctypes.c_int
    lib.xmix_ceiling_mfma.restype = ctypes.c_int
    # invalid arguments are rejected before any device call
    assert lib.xmix_ceiling_read(None, ctypes.c_uint64(16), None, None) == 1
    assert lib.xmix_ceiling_mfma(0, None, None, None) == 1


def test_batched_calls_check_every_app_on_the_host(lib):
    """Fake (never dereferenced) device addresses: the batched encode and
    clamp refuse a bad count, and an app the per-app call would refuse,
    before anything is launched."""
    import paper_2607_22595_amd as px
    A = 0x100000
    rt = px.XmixRoute(0x10000, 0x20000, 0x30000, 256, 4)
    good = px.XmixSaeDict(A, 65536, 4096, px.XMIX_SAE_DICT_TILED)
    bad = px.XmixSaeDict(A, 65536, 4096, 0)

    def app(bit=0, dct=good, k=64, ws_bytes=1 << 40, ring=None):
        return px.XmixSaeApp(bit, ctypes.pointer(dct), A, A, A, k, A, A, A, ws_bytes, ring, bit)

    enc = lib.xmix_sae_encode_topk_multi
    enc.restype = ctypes.c_int
    enc.argtypes = None

    def call(apps, n=None):
        arr = (px.XmixSaeApp * max(1, len(apps)))(*apps)
        return enc(ctypes.c_void_p(A), 4096, ctypes.byref(rt), len(apps) if n is None else n,
                   arr, ctypes.c_void_p(A), 0, None)
    assert call([app()], n=0) == 1
    assert call([app()] * 33) == 1                    # more than 32 apps
    assert call([app(), app(1, dct=bad)]) == 1         # a dictionary without its tag
    assert call([app(), app(bit=4)]) == 1              # bit outside the route's apps
    assert call([app(), app(k=65)]) == 1
    assert call([app(), app(ws_bytes=16)]) == 3        # workspace too small
    ring = px.XmixRing(A, A, 8, 16 + 6 * 64)
    arr = (px.XmixSaeApp * 1)(app(ring=ctypes.pointer(ring)))
    assert enc(ctypes.c_void_p(A), 4096, ctypes.byref(rt), 1, arr, None, 0, None) == 1  # no req
    clamp = lib.xmix_sae_clamp_decode_multi
    clamp.restype = ctypes.c_int
    clamp.argtypes = None

    def capp(bit=0, k=64, n_clamp=4):
        return px.XmixSaeClampApp(bit, A, A, k, A, 65536, A, A, n_clamp, None)
    carr = (px.XmixSaeClampApp * 2)(capp(), capp(n_clamp=17))
    assert clamp(ctypes.c_void_p(A), 4096, ctypes.byref(rt), 2, carr, None) == 1
    carr = (px.XmixSaeClampApp * 2)(capp(), capp(bit=7))
    assert clamp(ctypes.c_void_p(A), 4096, ctypes.byref(rt), 2, carr, None) == 1
    assert clamp(ctypes.c_void_p(A), 4096, ctypes.byref(rt), 0, carr, None) == 1
