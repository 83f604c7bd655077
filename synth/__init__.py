"""Seeded synthetic workloads for the per-layer MI hook step.

This module only draws inputs: activations, steering vectors, probe weights,
SAE dictionaries, per-request subscriptions and request layouts.  It holds
none of the hook step's arithmetic and is the one piece of code that both
the CPU oracle (through the tests) and the GPU path consume.

The paper's served models and ShareGPT traffic (Sec. 5, "Workload") are not
used: every tensor is drawn from a counter-based generator (SplitMix64 plus
Box-Muller, see ``gen.c``) with the shapes of the models the paper serves
(Llama-3.1-8B-like width 4096, a 70B-like width 8192).  A tensor is named by a
string such as ``"c3/sae0/W_enc"``; its stream key is FNV-1a of that name
mixed with the seed, so every tensor is independent of every other and of
the order in which they are drawn.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    u64, i64, dbl = ctypes.c_uint64, ctypes.c_int64, ctypes.c_double
    vp = ctypes.c_void_p
    lib.synth_normal_bf16.argtypes = [u64, i64, dbl, dbl, vp, i64, vp]
    lib.synth_normal_f32.argtypes = [u64, i64, dbl, dbl, vp, i64, vp]
    lib.synth_uniform_f32.argtypes = [u64, i64, dbl, dbl, vp]
    lib.synth_uniform_f64.argtypes = [u64, i64, vp]
    lib.synth_bits.argtypes = [u64, i64, vp]
    lib.synth_rownorm_bf16.argtypes = [vp, i64, i64, vp]
    lib.synth_bf16_from_double.argtypes = [dbl]
    lib.synth_bf16_from_double.restype = ctypes.c_uint16
    for name in ("synth_normal_bf16", "synth_normal_f32", "synth_uniform_f32",
                 "synth_uniform_f64", "synth_bits", "synth_rownorm_bf16"):
        getattr(lib, name).restype = None
    _lib = lib
    return lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


_MASK64 = (1 << 64) - 1


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def stream_key(name: str, seed: int = 0) -> int:
    """64-bit stream key of a named tensor: FNV-1a(name) mixed with the seed."""
    hsh = 0xCBF29CE484222325
    for byte in name.encode():
        hsh ^= byte
        hsh = (hsh * 0x100000001B3) & _MASK64
    return _mix((hsh + seed * 0x9E3779B97F4A7C15) & _MASK64)


# ----------------------------------------------------------------- primitives

def normal_bf16(name, shape, std, mean=0.0, chan_scale=None, seed=0):
    """bf16 bits (uint16) of mean + std * N(0, 1), rounded to nearest even.

    ``chan_scale`` (length = last dim) multiplies the std per channel."""
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    cs = None if chan_scale is None else np.ascontiguousarray(chan_scale, dtype=np.float64)
    _load().synth_normal_bf16(stream_key(name, seed), n, float(mean), float(std),
                              None if cs is None else _ptr(cs),
                              1 if cs is None else cs.size, _ptr(out))
    return out.reshape(shape)


def normal_f32(name, shape, std, mean=0.0, chan_scale=None, seed=0):
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    cs = None if chan_scale is None else np.ascontiguousarray(chan_scale, dtype=np.float64)
    _load().synth_normal_f32(stream_key(name, seed), n, float(mean), float(std),
                             None if cs is None else _ptr(cs),
                             1 if cs is None else cs.size, _ptr(out))
    return out.reshape(shape)


def uniform_f32(name, shape, lo, hi, seed=0):
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    _load().synth_uniform_f32(stream_key(name, seed), n, float(lo), float(hi), _ptr(out))
    return out.reshape(shape)


def uniform01(name, n, seed=0):
    out = np.empty(int(n), dtype=np.float64)
    _load().synth_uniform_f64(stream_key(name, seed), int(n), _ptr(out))
    return out


def randint(name, n, lo, hi, seed=0):
    """n integers uniform in [lo, hi] (inclusive)."""
    u = uniform01(name, n, seed)
    return (lo + np.floor(u * (hi - lo + 1))).astype(np.int64)


def permutation(name, n, seed=0):
    """A seeded permutation of range(n) (Fisher-Yates, Durstenfeld form)."""
    u = uniform01(name, max(n - 1, 0), seed)
    p = np.arange(n, dtype=np.int64)
    for i in range(n - 1, 0, -1):
        j = int(u[n - 1 - i] * (i + 1))
        p[i], p[j] = p[j], p[i]
    return p


def rownorm_bf16(W: np.ndarray) -> np.ndarray:
    """Rows of a bf16 matrix scaled to unit L2 norm (fp64 norm), rounded to bf16."""
    W = np.ascontiguousarray(W, dtype=np.uint16)
    out = np.empty_like(W)
    _load().synth_rownorm_bf16(_ptr(W), W.shape[0], W.shape[1], _ptr(out))
    return out


def bf16_from_double(x: float) -> int:
    return int(_load().synth_bf16_from_double(float(x)))


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bits to float32 values (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------------ workloads

@dataclass
class SteerApp:
    bit: int
    v: np.ndarray            # [d], bf16 bits or float32


@dataclass
class ProbeApp:
    bit: int
    w: np.ndarray            # [d], bf16 bits or float32
    b: float                 # fp32 bias
    mode: str                # "token", "mean" or "last"


@dataclass
class SaeApp:
    bit: int
    m: int
    k: int
    W_enc: np.ndarray        # [m, d] bf16 bits, latent-major
    b_enc: np.ndarray        # [m] bf16 bits
    b_dec: np.ndarray        # [d] bf16 bits
    W_dec: Optional[np.ndarray] = None      # [m, d] bf16 bits (clamp apps)
    clamp_ids: Optional[np.ndarray] = None  # int32 [n_clamp]
    clamp_vals: Optional[np.ndarray] = None  # float32 [n_clamp]
    ring_capacity: int = 0   # > 0: the encoded rows are read back into a ring


@dataclass
class Layer:
    layer_id: int
    h: np.ndarray            # [T_max, d] bf16 bits or float32
    steer: List[SteerApp] = field(default_factory=list)
    probes: List[ProbeApp] = field(default_factory=list)
    saes: List[SaeApp] = field(default_factory=list)


@dataclass
class Workload:
    name: str
    dtype: str               # "bf16" or "f32"
    d: int
    T_max: int
    T_valid: int
    R_max: int
    n_apps: int
    req: np.ndarray          # int32 [T_max]; -1 marks padding
    sub: np.ndarray          # uint32 [R_max]
    alpha: np.ndarray        # float32 [R_max, n_steer], shared by all layers
    layers: List[Layer]
    cu_seqlens: Optional[np.ndarray] = None   # int32 [R_max + 1]
    description: str = ""

    @property
    def n_steer(self):
        return len(self.layers[0].steer) if self.layers else 0


def _outlier_scale(cfg, d, n_out, seed):
    """Per-channel std multipliers: n_out fixed channels x20, the rest x1."""
    scale = np.ones(d, dtype=np.float64)
    if n_out:
        ids = permutation(f"{cfg}/outlier_channels", d, seed)[:n_out]
        scale[ids] = 20.0
    return scale


def _bern_sub(cfg, R, bits, p, seed):
    sub = np.zeros(R, dtype=np.uint32)
    for bit in bits:
        u = uniform01(f"{cfg}/sub/bit{bit}", R, seed)
        sub |= (u < p).astype(np.uint32) << np.uint32(bit)
    return sub


def ragged_lengths(cfg, R, total, lo, hi, seed=0, max_tries=100000):
    """R lengths in [lo, hi] summing to `total`: draw the first R-1 iid
    uniform in [lo, hi] and redraw all of them until the remainder also lies
    in [lo, hi] (seeded rejection)."""
    for attempt in range(max_tries):
        first = randint(f"{cfg}/lengths/try{attempt}", R - 1, lo, hi, seed)
        last = total - int(first.sum())
        if lo <= last <= hi:
            return np.concatenate([first, [last]]).astype(np.int64)
    raise ValueError("no feasible ragged layout")


def make_c1(seed=0, d=256, T=16, R=4):
    """Toy, fp32, 1 layer: app A (bit 0) steering with alpha 4.0 for requests
    {0, 2}; app B (bit 1) logistic probe with b = 0 for requests {1, 2, 3}."""
    cfg = "c1"
    req = randint(f"{cfg}/req", T, 0, R - 1, seed).astype(np.int32)
    sub = np.zeros(R, dtype=np.uint32)
    for r in (0, 2):
        if r < R:
            sub[r] |= 1
    for r in (1, 2, 3):
        if r < R:
            sub[r] |= 2
    h = normal_f32(f"{cfg}/L0/h", (T, d), 1.0, seed=seed)
    v = normal_f32(f"{cfg}/L0/steer0/v", (d,), 1.0 / np.sqrt(d), seed=seed)
    w = normal_f32(f"{cfg}/L0/probe0/w", (d,), 1.0 / np.sqrt(d), seed=seed)
    alpha = np.full((R, 1), 4.0, dtype=np.float32)
    layer = Layer(0, h, [SteerApp(0, v)], [ProbeApp(1, w, 0.0, "token")], [])
    return Workload(cfg, "f32", d, T, T, R, 2, req, sub, alpha, [layer],
                    description=f"toy fp32 d={d} T={T} R={R}")


def make_c2(seed=0, d=4096, T=256, n_layers=4, p=0.3, n_outliers=8):
    """Decode step, Llama-8B-shaped: one token per request, 4 hooked layers,
    bits 0-3 steering (alpha ~ U[-8, 8] per request and app), bits 4-7
    per-token probes; each (request, app) subscribed with probability p."""
    cfg = "c2"
    R = T
    req = np.arange(T, dtype=np.int32)
    sub = _bern_sub(cfg, R, range(8), p, seed)
    alpha = uniform_f32(f"{cfg}/alpha", (R, 4), -8.0, 8.0, seed)
    scale = _outlier_scale(cfg, d, n_outliers, seed)
    layers = []
    for L in range(n_layers):
        h = normal_bf16(f"{cfg}/L{L}/h", (T, d), 1.0, chan_scale=scale, seed=seed)
        steer = [SteerApp(s, normal_bf16(f"{cfg}/L{L}/steer{s}/v", (d,), 1 / np.sqrt(d), seed=seed))
                 for s in range(4)]
        probes = []
        for q in range(4):
            w = normal_bf16(f"{cfg}/L{L}/probe{q}/w", (d,), 1 / np.sqrt(d), seed=seed)
            b = float(normal_f32(f"{cfg}/L{L}/probe{q}/b", (1,), np.sqrt(0.1), seed=seed)[0])
            probes.append(ProbeApp(4 + q, w, b, "token"))
        layers.append(Layer(L, h, steer, probes, []))
    return Workload(cfg, "bf16", d, T, T, R, 8, req, sub, alpha, layers,
                    description=f"decode d={d} T=R={T} layers={n_layers}")


def _sae(cfg, tag, bit, d, m, k, seed, decoder=False):
    W = normal_bf16(f"{cfg}/{tag}/W_enc", (m, d), 1 / np.sqrt(d), seed=seed)
    b_enc = normal_bf16(f"{cfg}/{tag}/b_enc", (m,), 0.1, seed=seed)
    b_dec = normal_bf16(f"{cfg}/{tag}/b_dec", (d,), 0.1, seed=seed)
    app = SaeApp(bit, m, k, W, b_enc, b_dec)
    if decoder:
        app.W_dec = rownorm_bf16(W)
    return app


def make_c3(seed=0, d=4096, m=65536, k=64, T=256, n_sub=None, ring_capacity=256,
            n_outliers=8):
    """Decode-shaped SAE encode: one token per request, exactly half of the
    requests subscribed (seeded permutation), encoded rows read back into a
    ring of fixed capacity."""
    cfg = "c3"
    R = T
    if n_sub is None:
        n_sub = T // 2
    req = np.arange(T, dtype=np.int32)
    sub = np.zeros(R, dtype=np.uint32)
    sub[permutation(f"{cfg}/subscribed", R, seed)[:n_sub]] = 1
    scale = _outlier_scale(cfg, d, n_outliers, seed)
    h = normal_bf16(f"{cfg}/L0/h", (T, d), 1.0, chan_scale=scale, seed=seed)
    sae = _sae(cfg, "sae0", 0, d, m, k, seed)
    sae.ring_capacity = ring_capacity
    alpha = np.zeros((R, 0), dtype=np.float32)
    return Workload(cfg, "bf16", d, T, T, R, 1, req, sub, alpha, [Layer(0, h, [], [], [sae])],
                    description=f"decode SAE d={d} m={m} k={k} T={T} T_sub={n_sub}")


def make_c4(seed=0, d=4096, T=8192, R=16, len_lo=128, len_hi=1024, m=131072, k=32,
            n_outliers=8, n_last=0):
    """Prefill chunk: ragged requests in contiguous spans; bit 0 SAE encode on
    every token, bits 1-4 per-token probes, bits 5-8 mean-pooled probes, and
    (n_last > 0) bits 9.. last-token probes; every request subscribes to
    every app."""
    cfg = "c4"
    lens = ragged_lengths(cfg, R, T, len_lo, len_hi, seed)
    cu = np.zeros(R + 1, dtype=np.int32)
    cu[1:] = np.cumsum(lens)
    req = np.repeat(np.arange(R, dtype=np.int32), lens).astype(np.int32)
    n_apps = 9 + n_last
    sub = np.full(R, (1 << n_apps) - 1, dtype=np.uint32)
    scale = _outlier_scale(cfg, d, n_outliers, seed)
    h = normal_bf16(f"{cfg}/L0/h", (T, d), 1.0, chan_scale=scale, seed=seed)
    probes = []
    for q in range(8):
        w = normal_bf16(f"{cfg}/L0/probe{q}/w", (d,), 1 / np.sqrt(d), seed=seed)
        b = float(normal_f32(f"{cfg}/L0/probe{q}/b", (1,), np.sqrt(0.1), seed=seed)[0])
        probes.append(ProbeApp(1 + q, w, b, "token" if q < 4 else "mean"))
    for q in range(n_last):
        w = normal_bf16(f"{cfg}/L0/last{q}/w", (d,), 1 / np.sqrt(d), seed=seed)
        b = float(normal_f32(f"{cfg}/L0/last{q}/b", (1,), np.sqrt(0.1), seed=seed)[0])
        probes.append(ProbeApp(9 + q, w, b, "last"))
    sae = _sae(cfg, "sae0", 0, d, m, k, seed)
    alpha = np.zeros((R, 0), dtype=np.float32)
    return Workload(cfg, "bf16", d, T, T, R, n_apps, req, sub, alpha,
                    [Layer(0, h, [], probes, [sae])],
                    cu_seqlens=cu,
                    description=f"prefill d={d} T={T} R={R} m={m} k={k}")


def make_c5(seed=0, d=8192, T=512, m=65536, k=64, p=0.2, n_steer=16, n_probe=8, n_clamp_apps=8,
            n_clamp=4, clamp_value=10.0, n_outliers=8):
    """Decode step, 70B-shaped: 32 apps per request with probability p each;
    bits 0-15 steering, 16-23 per-token probes, 24-31 SAE clamp apps, each
    with its own dictionary (decoder = row-normalised encoder) and 4 clamped
    feature ids set to a fixed value."""
    cfg = "c5"
    R = T
    n_apps = n_steer + n_probe + n_clamp_apps
    req = np.arange(T, dtype=np.int32)
    sub = _bern_sub(cfg, R, range(n_apps), p, seed)
    alpha = uniform_f32(f"{cfg}/alpha", (R, n_steer), -8.0, 8.0, seed)
    scale = _outlier_scale(cfg, d, n_outliers, seed)
    h = normal_bf16(f"{cfg}/L0/h", (T, d), 1.0, chan_scale=scale, seed=seed)
    steer = [SteerApp(s, normal_bf16(f"{cfg}/L0/steer{s}/v", (d,), 1 / np.sqrt(d), seed=seed))
             for s in range(n_steer)]
    probes = []
    for q in range(n_probe):
        w = normal_bf16(f"{cfg}/L0/probe{q}/w", (d,), 1 / np.sqrt(d), seed=seed)
        b = float(normal_f32(f"{cfg}/L0/probe{q}/b", (1,), np.sqrt(0.1), seed=seed)[0])
        probes.append(ProbeApp(n_steer + q, w, b, "token"))
    saes = []
    for c in range(n_clamp_apps):
        sae = _sae(cfg, f"sae{c}", n_steer + n_probe + c, d, m, k, seed, decoder=True)
        sae.clamp_ids = np.sort(permutation(f"{cfg}/sae{c}/clamp_ids", m, seed)[:n_clamp]).astype(np.int32)
        sae.clamp_vals = np.full(n_clamp, clamp_value, dtype=np.float32)
        saes.append(sae)
    return Workload(cfg, "bf16", d, T, T, R, n_apps, req, sub, alpha,
                    [Layer(0, h, steer, probes, saes)],
                    description=f"decode d={d} T=R={T} apps={n_apps} m={m} k={k}")


MAKERS = {"c1": make_c1, "c2": make_c2, "c3": make_c3, "c4": make_c4, "c5": make_c5}


def make(name: str, **kw) -> Workload:
    return MAKERS[name](**kw)
