"""Python binding of libxmix, the MI355X (gfx950) per-layer MI hook step.

Argument marshalling only: every function below checks shapes and dtypes,
takes device pointers and the current HIP stream from torch tensors, and
calls the C entry point of the same name (declared in include/xmix.h).
All arithmetic runs in the library's HIP kernels.  There is no fallback:
importing this package fails if the built library is missing.

bf16 data is carried in ``torch.bfloat16`` tensors (raw bits on the C
side).  Route and ring descriptors own the device buffers the C structs
point to.
"""
from __future__ import annotations

import ctypes
import gc
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libxmix.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -c 'import __graft_entry__ as g; g.build()' or "
        "python paper_2607_22595_amd/build.py)")

_lib = ctypes.CDLL(LIB_PATH)

XMIX_OK, XMIX_E_INVAL, XMIX_E_UNSUPPORTED, XMIX_E_WORKSPACE, XMIX_E_LAUNCH = range(5)
XMIX_F32, XMIX_BF16 = 0, 1
XMIX_PROBE_TOKEN, XMIX_PROBE_MEAN, XMIX_PROBE_LAST = 0, 1, 2
XMIX_ERR_REQUEST_RANGE, XMIX_ERR_T_VALID = 1, 2
MAX_APPS, MAX_TOPK, MAX_CLAMP, MAX_SEGMENTS = 32, 64, 16, 4


class XmixRoute(ctypes.Structure):
    _fields_ = [("tok_mask", ctypes.c_void_p), ("app_count", ctypes.c_void_p),
                ("app_tokens", ctypes.c_void_p), ("T_max", ctypes.c_int32),
                ("n_apps", ctypes.c_int32)]


class XmixRing(ctypes.Structure):
    _fields_ = [("slots", ctypes.c_void_p), ("head", ctypes.c_void_p),
                ("capacity", ctypes.c_int32), ("row_bytes", ctypes.c_int32)]


XMIX_SAE_DICT_TILED = 0x31504D58


class XmixSaeDict(ctypes.Structure):
    _fields_ = [("pieces", ctypes.c_void_p), ("m", ctypes.c_int32), ("d", ctypes.c_int32),
                ("layout", ctypes.c_uint32)]


_vp, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
_dp = ctypes.POINTER(XmixSaeDict)


class XmixSaeApp(ctypes.Structure):
    _fields_ = [("app_bit", _i32), ("dict", _dp), ("b_enc", _vp), ("b_dec", _vp),
                ("c_fold", _vp), ("k", _i32), ("idx_out", _vp), ("val_out", _vp), ("ws", _vp),
                ("ws_bytes", _sz), ("ring", ctypes.POINTER(XmixRing)), ("app_id", _i32)]


class XmixSaeClampApp(ctypes.Structure):
    _fields_ = [("app_bit", _i32), ("idx", _vp), ("val", _vp), ("k", _i32), ("W_dec", _vp),
                ("m", _i32), ("clamp_ids", _vp), ("clamp_vals", _vp), ("n_clamp", _i32),
                ("delta_out", _vp)]


_st = ctypes.c_int
_sigs = {
    "xmix_status_string": ([_st], ctypes.c_char_p),
    "xmix_version": ([], ctypes.c_char_p),
    "xmix_route_build": ([_vp, _vp, _vp, _i32, ctypes.POINTER(XmixRoute), _vp, _vp], _st),
    "xmix_route_gate": ([ctypes.POINTER(XmixRoute), _i32, _vp, _vp, _i32, _i32, _vp, _vp], _st),
    "xmix_route_trigger": ([ctypes.POINTER(XmixRoute), _i32, _vp, _vp, _i32, _vp], _st),
    "xmix_graph_begin": ([_vp], _st),
    "xmix_graph_end": ([_vp, ctypes.POINTER(ctypes.c_void_p)], _st),
    "xmix_graph_kernel_nodes": ([_vp], _i32),
    "xmix_graph_redirect": ([_vp, _vp, _vp, ctypes.POINTER(ctypes.c_int32)], _st),
    "xmix_graph_launch": ([_vp, _vp], _st),
    "xmix_graph_destroy": ([_vp], None),
    "xmix_router_write": ([_vp, _st, _i32, ctypes.POINTER(XmixRoute), _vp, _vp, _i32, _vp],
                          _st),
    "xmix_steer_apply": ([_vp, _st, _i32, ctypes.POINTER(XmixRoute), _vp, _vp, _vp, _vp, _i32,
                          _i32, _vp], _st),
    "xmix_steer_probe": ([_vp, _st, _i32, ctypes.POINTER(XmixRoute), _vp, _vp, _vp, _vp, _i32,
                          _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp], _st),
    "xmix_route_steer_probe": ([_vp, _vp, _vp, _i32, ctypes.POINTER(XmixRoute), _vp, _vp, _st,
                                _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp, _i32, _vp, _vp, _vp],
                               _st),
    "xmix_probe_workspace": ([_i32, _i32, _i32], _sz),
    "xmix_probe_score": ([_vp, _st, _i32, ctypes.POINTER(XmixRoute), _vp, _vp, _vp, _i32, _i32,
                          _vp, _i32, _vp, _vp, _vp, _sz, _vp], _st),
    "xmix_sae_encode_workspace": ([_i32, _i32, _i32, _i32], _sz),
    "xmix_sae_encode_topk": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _dp, _vp, _vp, _vp,
                              _i32, _vp, _vp, _vp, _sz, _vp], _st),
    "xmix_sae_encode_topk_noalloc": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _dp, _vp,
                                      _vp, _vp, _i32, _vp, _vp, _vp], _st),
    "xmix_sae_encode_candidates": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _dp, _vp, _vp,
                                    _vp, _i32, _vp, _sz, _vp], _st),
    "xmix_route_sae_encode_candidates": ([_vp, _vp, _vp, _i32, ctypes.POINTER(XmixRoute), _vp,
                                          _vp, _i32, _i32, _dp, _vp, _vp, _vp, _i32, _vp, _sz,
                                          _vp], _st),
    "xmix_sae_merge_topk": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _dp, _vp, _i32, _vp,
                             _vp, _vp, _sz, _vp], _st),
    "xmix_sae_encode_topk_ring": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _dp, _vp, _vp,
                                   _vp, _i32, _vp, _vp, _vp, _sz, _vp, _i32, _i32,
                                   ctypes.POINTER(XmixRing), _vp], _st),
    "xmix_sae_merge_topk_ring": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _dp, _vp, _i32,
                                  _vp, _vp, _vp, _sz, _vp, _i32, _i32,
                                  ctypes.POINTER(XmixRing), _vp], _st),
    "xmix_sae_encode_topk_multi": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32,
                                    ctypes.POINTER(XmixSaeApp), _vp, _i32, _vp], _st),
    "xmix_route_sae_encode_topk_multi": ([_vp, _vp, _vp, _i32, ctypes.POINTER(XmixRoute), _vp,
                                          _vp, _i32, _i32, ctypes.POINTER(XmixSaeApp), _i32,
                                          _vp], _st),
    "xmix_sae_clamp_decode_multi": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32,
                                     ctypes.POINTER(XmixSaeClampApp), _vp], _st),
    "xmix_sae_pack_encoder": ([_vp, _i32, _i32, _vp, _dp, _vp], _st),
    "xmix_sae_fold_bias": ([_dp, _vp, _vp, _vp, _vp], _st),
    "xmix_sae_clamp_decode": ([_vp, _i32, ctypes.POINTER(XmixRoute), _i32, _vp, _vp, _i32, _vp,
                               _i32, _vp, _vp, _i32, _vp, _vp], _st),
    "xmix_readback_compact": ([_vp, _vp, _i32, ctypes.POINTER(XmixRoute), _i32, _vp, _i32, _i32,
                               ctypes.POINTER(XmixRing), _vp], _st),
}
for _name, (_args, _res) in _sigs.items():
    _fn = getattr(_lib, _name)
    _fn.argtypes = _args
    _fn.restype = _res

EXPORTED = tuple(_sigs)


class XmixError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = _lib.xmix_status_string(status).decode()
        super().__init__(f"{fn}: {msg} (status {status})")
        self.status = status


def _check(fn: str, status: int) -> None:
    if status != XMIX_OK:
        raise XmixError(fn, status)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return XMIX_BF16
    if t.dtype == torch.float32:
        return XMIX_F32
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def version() -> str:
    return _lib.xmix_version().decode()


# ---------------------------------------------------------------- descriptors

class Route:
    """Device routing table of one hook step (owns its buffers)."""

    def __init__(self, T_max: int, n_apps: int, device="cuda"):
        if not (1 <= n_apps <= MAX_APPS):
            raise ValueError("n_apps must be in [1, 32]")
        self.T_max, self.n_apps = int(T_max), int(n_apps)
        self.tok_mask = torch.zeros(T_max, dtype=torch.int32, device=device)
        self.app_count = torch.zeros(n_apps, dtype=torch.int32, device=device)
        self.app_tokens = torch.full((n_apps, T_max), -1, dtype=torch.int32, device=device)
        self.struct = XmixRoute(self.tok_mask.data_ptr(), self.app_count.data_ptr(),
                                self.app_tokens.data_ptr(), self.T_max, self.n_apps)


class Ring:
    """Device readback ring: slots [capacity, row_bytes] and head [2] (uint64)."""

    def __init__(self, capacity: int, row_bytes: int, device="cuda"):
        self.capacity, self.row_bytes = int(capacity), int(row_bytes)
        self.slots = torch.zeros((capacity, row_bytes), dtype=torch.uint8, device=device)
        self.head = torch.zeros(2, dtype=torch.int64, device=device)
        self.struct = XmixRing(self.slots.data_ptr(), self.head.data_ptr(), self.capacity,
                               self.row_bytes)


# ------------------------------------------------------------------ entries

def xmix_route_build(req_of_token, T_valid, sub_mask, route: Route, err_word, stream=None):
    """req_of_token int32 [T_max]; T_valid int32 [1]; sub_mask int32 [R_max]
    (uint32 bit patterns); err_word int32 [1] (bits ORed in)."""
    assert req_of_token.dtype == torch.int32 and req_of_token.numel() == route.T_max
    assert T_valid.dtype == torch.int32 and sub_mask.dtype == torch.int32
    _check("xmix_route_build", _lib.xmix_route_build(
        _ptr(req_of_token), _ptr(T_valid), _ptr(sub_mask), sub_mask.numel(),
        ctypes.byref(route.struct), _ptr(err_word), _stream(stream)))


def xmix_route_gate(route: Route, app_bit: int, signal, threshold, signal_bit: int = -1,
                    req_of_token=None, stream=None):
    """Activation-driven conditional write: keep app `app_bit` only on tokens
    whose signal (fp32 [T_max] per token, or [R] per request with
    req_of_token) is >= the device scalar `threshold`."""
    assert signal.dtype == torch.float32 and threshold.dtype == torch.float32
    _check("xmix_route_gate", _lib.xmix_route_gate(
        ctypes.byref(route.struct), app_bit, _ptr(signal), _ptr(req_of_token), signal.numel(),
        signal_bit, _ptr(threshold), _stream(stream)))


def xmix_route_trigger(route: Route, app_bit: int, token_ids, vocab_bits, vocab_size: int,
                       stream=None):
    """Token-driven conditional write: keep app `app_bit` only on tokens whose
    id (int32 [T_max]) is set in the trigger bitmap (int32 words)."""
    assert token_ids.dtype == torch.int32 and vocab_bits.numel() * 32 >= vocab_size
    _check("xmix_route_trigger", _lib.xmix_route_trigger(
        ctypes.byref(route.struct), app_bit, _ptr(token_ids), _ptr(vocab_bits), vocab_size,
        _stream(stream)))


def xmix_steer_apply(h, route: Route, req_of_token, vecs, app_bits: Sequence[int], alpha,
                     stream=None):
    """h [T_max, d] bf16/fp32 in place; vecs [n_steer, d] same dtype;
    alpha fp32 [R_max, n_steer]; app_bits: host list of route bits."""
    T_max, d = h.shape
    assert T_max == route.T_max and vecs.dtype == h.dtype and vecs.shape[-1] == d
    n = len(app_bits)
    assert alpha.dtype == torch.float32 and alpha.dim() == 2 and alpha.shape[1] == n
    bits = (ctypes.c_int32 * n)(*app_bits)
    _check("xmix_steer_apply", _lib.xmix_steer_apply(
        _ptr(h), _dt(h), d, ctypes.byref(route.struct), _ptr(req_of_token), _ptr(vecs), bits,
        _ptr(alpha), n, alpha.shape[0], _stream(stream)))


def xmix_steer_probe(h, route: Route, req_of_token, vecs, steer_bits: Sequence[int], alpha,
                     w, b, probe_bits: Sequence[int], logit_out, score_out, stream=None):
    """Token-mode probes and the steering add in one pass: the same results
    as xmix_probe_score(mode TOKEN) followed by xmix_steer_apply."""
    T_max, d = h.shape
    assert T_max == route.T_max and vecs.dtype == h.dtype and vecs.shape[-1] == d
    ns, npb = len(steer_bits), len(probe_bits)
    assert alpha.dtype == torch.float32 and alpha.dim() == 2 and alpha.shape[1] == ns
    assert w.dtype == h.dtype and w.shape == (npb, d) and b.dtype == torch.float32
    assert logit_out.shape == (npb, T_max) and score_out.shape == (npb, T_max)
    sb = (ctypes.c_int32 * ns)(*steer_bits)
    pb = (ctypes.c_int32 * npb)(*probe_bits)
    _check("xmix_steer_probe", _lib.xmix_steer_probe(
        _ptr(h), _dt(h), d, ctypes.byref(route.struct), _ptr(req_of_token), _ptr(vecs), sb,
        _ptr(alpha), ns, alpha.shape[0], _ptr(w), _ptr(b), pb, npb, _ptr(logit_out),
        _ptr(score_out), _stream(stream)))


def xmix_route_steer_probe(req_of_token, T_valid, sub_mask, route: Route, err_word, h, vecs,
                           steer_bits: Sequence[int], alpha, w, b, probe_bits: Sequence[int],
                           logit_out, score_out, stream=None):
    """Route build and the fused probes + steering pass in one launch (up to
    1024 token slots): the same results as xmix_route_build followed by
    xmix_steer_probe."""
    T_max, d = h.shape
    assert T_max == route.T_max and vecs.dtype == h.dtype and vecs.shape[-1] == d
    ns, npb = len(steer_bits), len(probe_bits)
    assert alpha.dtype == torch.float32 and alpha.dim() == 2 and alpha.shape[1] == ns
    assert w.dtype == h.dtype and w.shape == (npb, d) and b.dtype == torch.float32
    assert logit_out.shape == (npb, T_max) and score_out.shape == (npb, T_max)
    assert req_of_token.dtype == torch.int32 and req_of_token.numel() == T_max
    sb = (ctypes.c_int32 * ns)(*steer_bits)
    pb = (ctypes.c_int32 * npb)(*probe_bits)
    _check("xmix_route_steer_probe", _lib.xmix_route_steer_probe(
        _ptr(req_of_token), _ptr(T_valid), _ptr(sub_mask), sub_mask.numel(),
        ctypes.byref(route.struct), _ptr(err_word), _ptr(h), _dt(h), d, _ptr(vecs), sb,
        _ptr(alpha), ns, _ptr(w), _ptr(b), pb, npb, _ptr(logit_out), _ptr(score_out),
        _stream(stream)))


def xmix_router_write(logits, route: Route, app_bits: Sequence[int], offsets, stream=None):
    """logits [T_max, n_experts] bf16/fp32 in place; offsets fp32
    [n_router, n_experts] (-inf removes an expert); app_bits: host list of
    route bits, one per router app."""
    T_max, E = logits.shape
    assert T_max == route.T_max and logits.is_contiguous()
    n = len(app_bits)
    assert offsets.dtype == torch.float32 and tuple(offsets.shape) == (n, E)
    bits = (ctypes.c_int32 * n)(*app_bits)
    _check("xmix_router_write", _lib.xmix_router_write(
        _ptr(logits), _dt(logits), E, ctypes.byref(route.struct), bits, _ptr(offsets), n,
        _stream(stream)))


class Graph:
    """A sequence of library calls captured once on `stream` (xmix_graph_begin
    / xmix_graph_end) and replayed with launch().  redirect(old, new) points
    every kernel argument that holds tensor `old` at tensor `new` (same size
    and layout) through a kernel-node parameter update; it returns the
    number of arguments changed.  Nothing else may run on `stream` during
    the capture, and `record` must not synchronise or allocate."""

    def __init__(self, record, stream):
        if not isinstance(stream, torch.cuda.Stream):
            raise ValueError("capture needs a torch.cuda.Stream (not the null stream)")
        self.stream = stream
        self._h = ctypes.c_void_p()
        # An object collected during the capture (a torch CUDA graph, say)
        # could make a HIP call that is not allowed while the stream
        # captures: collect first and keep the collector off until the end.
        gc_was_on = gc.isenabled()
        gc.collect()
        gc.disable()
        try:
            _check("xmix_graph_begin", _lib.xmix_graph_begin(_stream(stream)))
            try:
                record()
            finally:
                st = _lib.xmix_graph_end(_stream(stream), ctypes.byref(self._h))
            _check("xmix_graph_end", st)
        finally:
            if gc_was_on:
                gc.enable()

    @property
    def kernel_nodes(self) -> int:
        return int(_lib.xmix_graph_kernel_nodes(self._h))

    def redirect(self, old, new) -> int:
        if old.numel() * old.element_size() != new.numel() * new.element_size():
            raise ValueError("redirect needs buffers of the same size")
        n = ctypes.c_int32(0)
        _check("xmix_graph_redirect", _lib.xmix_graph_redirect(self._h, _ptr(old), _ptr(new),
                                                               ctypes.byref(n)))
        return int(n.value)

    def launch(self, stream=None):
        _check("xmix_graph_launch", _lib.xmix_graph_launch(
            self._h, _stream(self.stream if stream is None else stream)))

    def close(self):
        if self._h:
            _lib.xmix_graph_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def probe_workspace(T_max: int, n_probe: int, mode: int) -> int:
    return int(_lib.xmix_probe_workspace(T_max, n_probe, mode))


def xmix_probe_score(h, route: Route, w, b, app_bits: Sequence[int], mode: int, logit_out,
                     score_out, cu_seqlens=None, ws=None, stream=None):
    """Token mode: outputs fp32 [n_probe, T_max].  Mean and last-token modes:
    outputs fp32 [n_probe, R_max] with cu_seqlens int32 [R_max + 1]."""
    T_max, d = h.shape
    n = len(app_bits)
    assert w.dtype == h.dtype and w.shape == (n, d) and b.dtype == torch.float32
    R_max = 0
    if mode in (XMIX_PROBE_MEAN, XMIX_PROBE_LAST):
        R_max = cu_seqlens.numel() - 1
        assert logit_out.shape == (n, R_max)
    else:
        assert logit_out.shape == (n, T_max)
    bits = (ctypes.c_int32 * n)(*app_bits)
    ws_bytes = 0 if ws is None else ws.numel() * ws.element_size()
    _check("xmix_probe_score", _lib.xmix_probe_score(
        _ptr(h), _dt(h), d, ctypes.byref(route.struct), _ptr(w), _ptr(b), bits, n, mode,
        _ptr(cu_seqlens), R_max, _ptr(logit_out), _ptr(score_out), _ptr(ws), ws_bytes,
        _stream(stream)))


def sae_encode_workspace(T_max: int, d: int, m: int, k: int) -> int:
    return int(_lib.xmix_sae_encode_workspace(T_max, d, m, k))


class SaeDict:
    """An encoder dictionary packed by xmix_sae_pack_encoder: the device
    buffer of m * d bf16 in the library's tiled layout (``packed``) and the
    C descriptor that points at it (``struct``)."""

    def __init__(self, packed: torch.Tensor, struct: XmixSaeDict):
        self.packed = packed
        self.struct = struct
        self.m, self.d = int(struct.m), int(struct.d)

    @property
    def nbytes(self) -> int:
        return self.packed.numel() * self.packed.element_size()

    def clone(self) -> "SaeDict":
        """A second device copy of the packed bytes with its own descriptor."""
        p = self.packed.clone()
        return SaeDict(p, XmixSaeDict(p.data_ptr(), self.m, self.d, self.struct.layout))

    def ref(self):
        return ctypes.byref(self.struct)


def _dict(W) -> SaeDict:
    if not isinstance(W, SaeDict):
        raise TypeError("the encoder dictionary must come from xmix_sae_pack_encoder")
    return W


def xmix_sae_pack_encoder(W_enc, W_packed=None, stream=None) -> SaeDict:
    """Row-major bf16 W_enc [m, d] -> the tiled layout the encode streams.
    Returns the packed dictionary (a new device buffer unless W_packed, a
    bf16 tensor of m * d elements, is given)."""
    m, d = W_enc.shape
    assert W_enc.dtype == torch.bfloat16
    if W_packed is None:
        W_packed = torch.empty_like(W_enc)
    assert W_packed.dtype == torch.bfloat16 and W_packed.numel() == m * d
    st = XmixSaeDict()
    _check("xmix_sae_pack_encoder", _lib.xmix_sae_pack_encoder(
        _ptr(W_enc), m, d, _ptr(W_packed), ctypes.byref(st), _stream(stream)))
    return SaeDict(W_packed, st)


def xmix_sae_fold_bias(W: SaeDict, b_enc, b_dec, c_fold, stream=None):
    W = _dict(W)
    assert c_fold.dtype == torch.float32 and c_fold.numel() == W.m
    _check("xmix_sae_fold_bias", _lib.xmix_sae_fold_bias(
        W.ref(), _ptr(b_enc), _ptr(b_dec), _ptr(c_fold), _stream(stream)))


def xmix_sae_encode_topk(h, route: Route, app_bit: int, W: SaeDict, b_enc, b_dec, c_fold,
                         k: int, idx_out, val_out, ws, stream=None):
    """h bf16 [T_max, d]; W the packed dictionary; c_fold fp32 [m] or None;
    idx_out int32 [T_max, k]; val_out bf16 [T_max, k]; ws uint8 workspace."""
    T_max, d = h.shape
    W = _dict(W)
    assert h.dtype == torch.bfloat16
    assert idx_out.dtype == torch.int32 and idx_out.shape == (T_max, k)
    assert val_out.dtype == torch.bfloat16 and val_out.shape == (T_max, k)
    ws_bytes = ws.numel() * ws.element_size()
    _check("xmix_sae_encode_topk", _lib.xmix_sae_encode_topk(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, W.ref(), _ptr(b_enc), _ptr(b_dec),
        _ptr(c_fold), k, _ptr(idx_out), _ptr(val_out), _ptr(ws), ws_bytes, _stream(stream)))


XMIX_STATIC_SCRATCH_BYTES = 16 << 20


def xmix_sae_encode_topk_noalloc(h, route: Route, app_bit: int, W: SaeDict, b_enc, b_dec,
                                 c_fold, k: int, idx_out, val_out, stream=None):
    """xmix_sae_encode_topk with the library's own per-GPU static workspace
    (no workspace argument, nothing allocated by the call)."""
    T_max, d = h.shape
    W = _dict(W)
    assert h.dtype == torch.bfloat16
    assert idx_out.dtype == torch.int32 and idx_out.shape == (T_max, k)
    assert val_out.dtype == torch.bfloat16 and val_out.shape == (T_max, k)
    _check("xmix_sae_encode_topk_noalloc", _lib.xmix_sae_encode_topk_noalloc(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, W.ref(), _ptr(b_enc), _ptr(b_dec),
        _ptr(c_fold), k, _ptr(idx_out), _ptr(val_out), _stream(stream)))


def xmix_sae_encode_topk_ring(h, route: Route, app_bit: int, W: SaeDict, b_enc, b_dec, c_fold,
                              k: int, idx_out, val_out, ws, req_of_token, layer_id: int,
                              app_id: int, ring: Ring, stream=None):
    """xmix_sae_encode_topk with the ring readback of (idx, val) rows fused
    into the merge; ring.row_bytes must be 16 + 6 k."""
    T_max, d = h.shape
    W = _dict(W)
    assert h.dtype == torch.bfloat16
    assert idx_out.dtype == torch.int32 and idx_out.shape == (T_max, k)
    assert val_out.dtype == torch.bfloat16 and val_out.shape == (T_max, k)
    assert req_of_token.dtype == torch.int32 and req_of_token.numel() == T_max
    _check("xmix_sae_encode_topk_ring", _lib.xmix_sae_encode_topk_ring(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, W.ref(), _ptr(b_enc), _ptr(b_dec),
        _ptr(c_fold), k, _ptr(idx_out), _ptr(val_out), _ptr(ws), ws.numel() * ws.element_size(),
        _ptr(req_of_token), layer_id, app_id, ctypes.byref(ring.struct), _stream(stream)))


def xmix_sae_merge_topk_ring(h, route: Route, app_bit: int, W: SaeDict, c_fold, k: int, idx_out,
                             val_out, ws, req_of_token, layer_id: int, app_id: int, ring: Ring,
                             stream=None):
    """Stage 2 of the encode with the fused ring readback."""
    T_max, d = h.shape
    W = _dict(W)
    _check("xmix_sae_merge_topk_ring", _lib.xmix_sae_merge_topk_ring(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, W.ref(), _ptr(c_fold), k,
        _ptr(idx_out), _ptr(val_out), _ptr(ws), ws.numel() * ws.element_size(),
        _ptr(req_of_token), layer_id, app_id, ctypes.byref(ring.struct), _stream(stream)))


def xmix_route_sae_encode_candidates(req_of_token, T_valid, sub_mask, route: Route, err_word, h,
                                     app_bit: int, W: SaeDict, b_enc, b_dec, c_fold, k: int, ws,
                                     stream=None):
    """Route build and the encode's candidates stage in one launch (up to
    1024 token slots): the same results as xmix_route_build followed by
    xmix_sae_encode_candidates."""
    T_max, d = h.shape
    W = _dict(W)
    assert T_max == route.T_max and h.dtype == torch.bfloat16
    _check("xmix_route_sae_encode_candidates", _lib.xmix_route_sae_encode_candidates(
        _ptr(req_of_token), _ptr(T_valid), _ptr(sub_mask), sub_mask.numel(),
        ctypes.byref(route.struct), _ptr(err_word), _ptr(h), d, app_bit, W.ref(),
        _ptr(b_enc), _ptr(b_dec), _ptr(c_fold), k, _ptr(ws), ws.numel() * ws.element_size(),
        _stream(stream)))


def xmix_sae_encode_candidates(h, route: Route, app_bit: int, W: SaeDict, b_enc, b_dec, c_fold,
                               k: int, ws, stream=None):
    """Stage 1 of the encode: per-slice top-k candidates into `ws`."""
    T_max, d = h.shape
    W = _dict(W)
    assert h.dtype == torch.bfloat16
    _check("xmix_sae_encode_candidates", _lib.xmix_sae_encode_candidates(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, W.ref(), _ptr(b_enc), _ptr(b_dec),
        _ptr(c_fold), k, _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def xmix_sae_merge_topk(h, route: Route, app_bit: int, W: SaeDict, c_fold, k: int, idx_out,
                        val_out, ws, stream=None):
    """Stage 2 of the encode: exact top-k per token from the candidates."""
    T_max, d = h.shape
    W = _dict(W)
    _check("xmix_sae_merge_topk", _lib.xmix_sae_merge_topk(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, W.ref(), _ptr(c_fold), k,
        _ptr(idx_out), _ptr(val_out), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def xmix_sae_clamp_decode(h, route: Route, app_bit: int, idx, val, W_dec, clamp_ids,
                          clamp_vals, delta_out=None, stream=None):
    T_max, d = h.shape
    k = idx.shape[1]
    m = W_dec.shape[0]
    assert h.dtype == torch.bfloat16 and W_dec.dtype == torch.bfloat16
    assert clamp_ids.dtype == torch.int32 and clamp_vals.dtype == torch.float32
    _check("xmix_sae_clamp_decode", _lib.xmix_sae_clamp_decode(
        _ptr(h), d, ctypes.byref(route.struct), app_bit, _ptr(idx), _ptr(val), k, _ptr(W_dec), m,
        _ptr(clamp_ids), _ptr(clamp_vals), clamp_ids.numel(), _ptr(delta_out), _stream(stream)))


class SaeApp:
    """One SAE app of a batched encode: the per-app arguments of
    xmix_sae_encode_topk (ring None) or xmix_sae_encode_topk_ring."""

    def __init__(self, app_bit: int, W: SaeDict, b_enc, b_dec, c_fold, k: int, idx_out,
                 val_out, ws, ring: Optional[Ring] = None, app_id: Optional[int] = None):
        self.app_bit, self.W, self.b_enc, self.b_dec, self.c_fold = app_bit, _dict(W), b_enc, \
            b_dec, c_fold
        self.k, self.idx_out, self.val_out, self.ws, self.ring = k, idx_out, val_out, ws, ring
        self.app_id = app_bit if app_id is None else app_id

    def struct(self, T_max: int) -> XmixSaeApp:
        assert self.idx_out.dtype == torch.int32 and self.idx_out.shape == (T_max, self.k)
        assert self.val_out.dtype == torch.bfloat16 and self.val_out.shape == (T_max, self.k)
        return XmixSaeApp(self.app_bit, ctypes.pointer(self.W.struct), _ptr(self.b_enc),
                          _ptr(self.b_dec), _ptr(self.c_fold), self.k, _ptr(self.idx_out),
                          _ptr(self.val_out), _ptr(self.ws),
                          self.ws.numel() * self.ws.element_size(),
                          ctypes.pointer(self.ring.struct) if self.ring is not None else None,
                          self.app_id)


def _sae_apps(apps: Sequence[SaeApp], T_max: int):
    arr = (XmixSaeApp * len(apps))(*[a.struct(T_max) for a in apps])
    return arr


def xmix_sae_encode_topk_multi(h, route: Route, apps: Sequence[SaeApp], req_of_token=None,
                               layer_id: int = 0, stream=None):
    """The SAE apps of one hook encoded together (results identical to one
    xmix_sae_encode_topk or _ring call per app)."""
    T_max, d = h.shape
    assert h.dtype == torch.bfloat16
    arr = _sae_apps(apps, T_max)
    _check("xmix_sae_encode_topk_multi", _lib.xmix_sae_encode_topk_multi(
        _ptr(h), d, ctypes.byref(route.struct), len(apps), arr, _ptr(req_of_token), layer_id,
        _stream(stream)))


def xmix_route_sae_encode_topk_multi(req_of_token, T_valid, sub_mask, route: Route, err_word, h,
                                     apps: Sequence[SaeApp], layer_id: int = 0, stream=None):
    """The batched encode with the step's routing built by its first launch."""
    T_max, d = h.shape
    assert T_max == route.T_max and h.dtype == torch.bfloat16
    arr = _sae_apps(apps, T_max)
    _check("xmix_route_sae_encode_topk_multi", _lib.xmix_route_sae_encode_topk_multi(
        _ptr(req_of_token), _ptr(T_valid), _ptr(sub_mask), sub_mask.numel(),
        ctypes.byref(route.struct), _ptr(err_word), _ptr(h), d, len(apps), arr, layer_id,
        _stream(stream)))


def xmix_sae_clamp_decode_multi(h, route: Route, apps: Sequence[tuple], stream=None):
    """apps: (app_bit, idx, val, W_dec, clamp_ids, clamp_vals[, delta_out]) per
    clamp app, applied in this order (h ends as after one
    xmix_sae_clamp_decode call per app)."""
    T_max, d = h.shape
    assert h.dtype == torch.bfloat16
    items = []
    for a in apps:
        bit, idx, val, W_dec, ids, vals = a[:6]
        delta = a[6] if len(a) > 6 else None
        assert W_dec.dtype == torch.bfloat16 and ids.dtype == torch.int32
        assert vals.dtype == torch.float32
        items.append(XmixSaeClampApp(bit, _ptr(idx), _ptr(val), idx.shape[1], _ptr(W_dec),
                                     W_dec.shape[0], _ptr(ids), _ptr(vals), ids.numel(),
                                     _ptr(delta)))
    arr = (XmixSaeClampApp * len(items))(*items)
    _check("xmix_sae_clamp_decode_multi", _lib.xmix_sae_clamp_decode_multi(
        _ptr(h), d, ctypes.byref(route.struct), len(items), arr, _stream(stream)))


def xmix_readback_compact(segments: Sequence[torch.Tensor], route: Route, app_bit: int,
                          req_of_token, layer_id: int, app_id: int, ring: Ring, stream=None):
    """segments: device tensors whose row t (dim 0) is copied verbatim."""
    n = len(segments)
    ptrs = (ctypes.c_void_p * n)(*[_ptr(s) for s in segments])
    sizes = (ctypes.c_int32 * n)(*[s[0].numel() * s.element_size() for s in segments])
    _check("xmix_readback_compact", _lib.xmix_readback_compact(
        ptrs, sizes, n, ctypes.byref(route.struct), app_bit, _ptr(req_of_token), layer_id,
        app_id, ctypes.byref(ring.struct), _stream(stream)))
