"""CPU oracle for the per-layer MI hook step (fp64, plain C loops).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg are the only callers.  The product path
(the HIP library and its Python binding) never imports this package, and
this package never imports the product.

Each wrapper below marshals numpy arrays into the C functions of
``oracle.c``; the arithmetic, and the passage of the paper each function
follows, is documented there.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64
    lib.oracle_round_bf16.argtypes = [ctypes.c_double]
    lib.oracle_round_bf16.restype = ctypes.c_uint16
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    lib.oracle_route.argtypes = [vp, i32, i32, vp, i32, i32, vp, vp, vp, vp]
    lib.oracle_steer.argtypes = [vp, ctypes.c_int, i32, i32, vp, vp, vp, vp, vp, i32]
    lib.oracle_router_write.argtypes = [vp, ctypes.c_int, i32, i32, vp, vp, vp, i32]
    lib.oracle_probe_token.argtypes = [vp, ctypes.c_int, i32, i32, vp, vp, vp, vp, i32, vp, vp]
    lib.oracle_probe_mean.argtypes = [vp, ctypes.c_int, i32, i32, vp, vp, vp, vp, i32, vp, i32, vp, vp]
    lib.oracle_route_gate.argtypes = [i32, vp, vp, vp, i32, vp, i32, vp, i32, i32, ctypes.c_float]
    lib.oracle_route_trigger.argtypes = [i32, vp, vp, vp, i32, vp, vp, i32]
    lib.oracle_probe_last.argtypes = [vp, ctypes.c_int, i32, i32, vp, vp, vp, vp, i32, vp, i32, vp, vp]
    lib.oracle_sae_pre.argtypes = [vp, i32, vp, vp, vp, i32, vp]
    lib.oracle_topk.argtypes = [vp, i32, i32, vp, vp, vp]
    lib.oracle_sae_encode.argtypes = [vp, i32, vp, i32, vp, vp, vp, i32, i32, vp, vp, vp, vp]
    lib.oracle_clamp_decode.argtypes = [vp, i32, i32, vp, i32, vp, vp, i32, vp, i32, vp, vp, i32, vp]
    lib.oracle_compact.argtypes = [vp, vp, i32, vp, i32, i32, vp, i32, i32, vp, i32, i32, vp]
    for n in ("oracle_route", "oracle_route_gate", "oracle_route_trigger", "oracle_steer", "oracle_probe_token", "oracle_probe_mean", "oracle_probe_last",
              "oracle_sae_pre", "oracle_topk", "oracle_sae_encode", "oracle_clamp_decode",
              "oracle_compact"):
        getattr(lib, n).restype = None
    _ = u64
    _lib = lib
    return lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a):
    return None if a is None else a.ctypes.data


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Threads the oracle's parallel loops use from now on."""
    _load().oracle_set_num_threads(int(n))


def round_bf16(x: float) -> int:
    """bf16 bits of x rounded to nearest, ties to even (from fp64)."""
    return int(_load().oracle_round_bf16(float(x)))


def bf16_to_f64(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def route(req, T_valid, sub, n_apps, R_max=None):
    """Returns (tok_mask u32[T_max], count i32[n_apps], app_tokens i32[n_apps,T_max], err)."""
    req = _c(req, np.int32)
    sub = _c(sub, np.uint32)
    T_max = req.size
    R_max = sub.size if R_max is None else R_max
    tok_mask = np.empty(T_max, np.uint32)
    count = np.empty(max(n_apps, 1), np.int32)
    app_tokens = np.empty((max(n_apps, 1), T_max), np.int32)
    err = np.zeros(1, np.uint32)
    _load().oracle_route(_p(req), int(T_valid), T_max, _p(sub), int(R_max), int(n_apps),
                         _p(tok_mask), _p(count), _p(app_tokens), _p(err))
    return tok_mask, count[:n_apps], app_tokens[:n_apps], int(err[0])


def route_gate(tok_mask, count, app_tokens, app_bit, signal, threshold, signal_bit=-1,
               req=None):
    """Activation-driven conditional write: narrows app `app_bit` of a route
    (tok_mask, count, app_tokens as returned by route()) to the tokens whose
    signal passes `threshold`; per-request signal when `req` is given.
    Returns new (tok_mask, count, app_tokens)."""
    tm = np.array(tok_mask, np.uint32, copy=True)
    T_max = tm.size
    n_apps = app_tokens.shape[0]
    cnt = np.array(count, np.int32, copy=True)
    lists = np.ascontiguousarray(np.array(app_tokens, np.int32, copy=True))
    sig = _c(signal, np.float32)
    per_req = req is not None
    reqv = _c(req, np.int32) if per_req else np.zeros(1, np.int32)
    _load().oracle_route_gate(T_max, _p(tm), _p(cnt), _p(lists), int(app_bit), _p(sig),
                              int(per_req), _p(reqv), int(sig.size), int(signal_bit),
                              ctypes.c_float(threshold))
    return tm, cnt[:n_apps], lists


def route_trigger(tok_mask, count, app_tokens, app_bit, token_ids, vocab_bits, vocab_size):
    """Token-driven conditional write: narrows app `app_bit` to the tokens whose
    id is in the trigger bitmap.  Returns new (tok_mask, count, app_tokens)."""
    tm = np.array(tok_mask, np.uint32, copy=True)
    T_max = tm.size
    n_apps = app_tokens.shape[0]
    cnt = np.array(count, np.int32, copy=True)
    lists = np.ascontiguousarray(np.array(app_tokens, np.int32, copy=True))
    _load().oracle_route_trigger(T_max, _p(tm), _p(cnt), _p(lists), int(app_bit),
                                 _p(_c(token_ids, np.int32)), _p(_c(vocab_bits, np.uint32)),
                                 int(vocab_size))
    return tm, cnt[:n_apps], lists


def steer(h, tok_mask, req, v, app_bits, alpha):
    """Returns the steered copy of h (same dtype: uint16 bf16 bits or float32)."""
    is_bf16 = h.dtype == np.uint16
    out = np.array(h, copy=True, order="C")
    T_max, d = out.shape
    v = _c(v, out.dtype).reshape(-1, d)
    n_steer = v.shape[0]
    alpha = _c(alpha, np.float32).reshape(-1, n_steer) if n_steer else np.zeros((1, 1), np.float32)
    _load().oracle_steer(_p(out), int(is_bf16), T_max, d, _p(_c(tok_mask, np.uint32)),
                         _p(_c(req, np.int32)), _p(v), _p(_c(app_bits, np.int32)), _p(alpha), n_steer)
    return out


def router_write(logits, tok_mask, app_bits, offsets):
    """Returns the written copy of the router logits [T_max, n_experts]
    (uint16 bf16 bits or float32); offsets float32 [n_router, n_experts]."""
    is_bf16 = logits.dtype == np.uint16
    out = np.array(logits, copy=True, order="C")
    T_max, E = out.shape
    off = _c(offsets, np.float32).reshape(-1, E)
    _load().oracle_router_write(_p(out), int(is_bf16), T_max, E, _p(_c(tok_mask, np.uint32)),
                                _p(_c(app_bits, np.int32)), _p(off), off.shape[0])
    return out


def probe_token(h, tok_mask, w, b, app_bits):
    """Returns (logit, score) as float64 [n_probe, T_max]; NaN where not written."""
    is_bf16 = h.dtype == np.uint16
    h = _c(h, h.dtype)
    T_max, d = h.shape
    w = _c(w, h.dtype).reshape(-1, d)
    n = w.shape[0]
    logit = np.full((n, T_max), np.nan)
    score = np.full((n, T_max), np.nan)
    _load().oracle_probe_token(_p(h), int(is_bf16), T_max, d, _p(_c(tok_mask, np.uint32)), _p(w),
                               _p(_c(b, np.float32)), _p(_c(app_bits, np.int32)), n,
                               _p(logit), _p(score))
    return logit, score


def probe_mean(h, tok_mask, w, b, app_bits, cu_seqlens):
    """Returns (logit, score) as float64 [n_probe, R]; NaN where not written."""
    is_bf16 = h.dtype == np.uint16
    h = _c(h, h.dtype)
    T_max, d = h.shape
    w = _c(w, h.dtype).reshape(-1, d)
    n = w.shape[0]
    cu = _c(cu_seqlens, np.int32)
    R = cu.size - 1
    logit = np.full((n, R), np.nan)
    score = np.full((n, R), np.nan)
    _load().oracle_probe_mean(_p(h), int(is_bf16), T_max, d, _p(_c(tok_mask, np.uint32)), _p(w),
                              _p(_c(b, np.float32)), _p(_c(app_bits, np.int32)), n, _p(cu), R,
                              _p(logit), _p(score))
    return logit, score


def probe_last(h, tok_mask, w, b, app_bits, cu_seqlens):
    """Returns (logit, score) as float64 [n_probe, R]; NaN where not written."""
    is_bf16 = h.dtype == np.uint16
    h = _c(h, h.dtype)
    T_max, d = h.shape
    w = _c(w, h.dtype).reshape(-1, d)
    n = w.shape[0]
    cu = _c(cu_seqlens, np.int32)
    R = cu.size - 1
    logit = np.full((n, R), np.nan)
    score = np.full((n, R), np.nan)
    _load().oracle_probe_last(_p(h), int(is_bf16), T_max, d, _p(_c(tok_mask, np.uint32)), _p(w),
                              _p(_c(b, np.float32)), _p(_c(app_bits, np.int32)), n, _p(cu), R,
                              _p(logit), _p(score))
    return logit, score


def sae_pre(h_row, W_enc, b_enc, b_dec):
    d = h_row.size
    m = W_enc.shape[0]
    pre = np.empty(m, np.float64)
    _load().oracle_sae_pre(_p(_c(h_row, np.uint16)), d, _p(_c(W_enc, np.uint16)),
                           _p(_c(b_enc, np.uint16)), _p(_c(b_dec, np.uint16)), m, _p(pre))
    return pre


def topk(pre, k):
    pre = _c(pre, np.float64)
    idx = np.empty(k, np.int32)
    ve = np.empty(k, np.float64)
    vb = np.empty(k, np.uint16)
    _load().oracle_topk(_p(pre), pre.size, int(k), _p(idx), _p(ve), _p(vb))
    return idx, ve, vb


def sae_encode(h, tokens, W_enc, b_enc, b_dec, k, want_pre=False):
    """Encode rows `tokens` of h.  Returns (idx i32[n,k], val bf16-bits u16[n,k],
    val_exact f64[n,k], pre f64[n,m] or None)."""
    h = _c(h, np.uint16)
    d = h.shape[1]
    tokens = _c(tokens, np.int32)
    n = tokens.size
    W_enc = _c(W_enc, np.uint16)
    m = W_enc.shape[0]
    idx = np.empty((n, k), np.int32)
    val = np.empty((n, k), np.uint16)
    ve = np.empty((n, k), np.float64)
    pre = np.empty((n, m), np.float64) if want_pre else None
    if n:
        _load().oracle_sae_encode(_p(h), d, _p(tokens), n, _p(W_enc), _p(_c(b_enc, np.uint16)),
                                  _p(_c(b_dec, np.uint16)), m, int(k), _p(idx), _p(val), _p(ve),
                                  _p(pre))
    return idx, val, ve, pre


def clamp_decode(h, tok_mask, app_bit, idx, val, W_dec, clamp_ids, clamp_vals, want_delta=False):
    """Returns (h', delta f64[T_max, d] or None).  idx/val are token-indexed [T_max, k]."""
    out = np.array(h, dtype=np.uint16, copy=True, order="C")
    T_max, d = out.shape
    idx = _c(idx, np.int32).reshape(T_max, -1)
    k = idx.shape[1]
    val = _c(val, np.uint16).reshape(T_max, k)
    W_dec = _c(W_dec, np.uint16)
    ids = _c(clamp_ids, np.int32)
    delta = np.full((T_max, d), np.nan) if want_delta else None
    _load().oracle_clamp_decode(_p(out), T_max, d, _p(_c(tok_mask, np.uint32)), int(app_bit),
                                _p(idx), _p(val), k, _p(W_dec), W_dec.shape[0], _p(ids),
                                _p(_c(clamp_vals, np.float32)), ids.size, _p(delta))
    return out, delta


def compact(segments, tok_mask, app_bit, req, layer_id, app_id, slots, head):
    """segments: list of uint8 arrays [T_max, seg_bytes].  slots: uint8
    [capacity, row_bytes] (updated copy returned).  Returns (slots, head)."""
    segs = [np.ascontiguousarray(s).view(np.uint8).reshape(s.shape[0], -1) for s in segments]
    T_max = segs[0].shape[0] if segs else np.asarray(tok_mask).size
    ptrs = (ctypes.c_void_p * max(len(segs), 1))(*[s.ctypes.data for s in segs])
    sizes = np.array([s.shape[1] for s in segs] or [0], np.int32)
    out = np.array(slots, dtype=np.uint8, copy=True, order="C")
    cap, row_bytes = out.shape
    hd = np.array([head], np.uint64)
    _load().oracle_compact(ctypes.cast(ptrs, ctypes.c_void_p), _p(sizes), len(segs),
                           _p(_c(tok_mask, np.uint32)), T_max, int(app_bit), _p(_c(req, np.int32)),
                           int(layer_id), int(app_id), _p(out), cap, row_bytes, _p(hd))
    return out, int(hd[0])
