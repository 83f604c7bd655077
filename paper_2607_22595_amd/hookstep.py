"""One hook step of a continuously batched forward pass, on the GPU.

``HookStep`` uploads a workload (activations per hooked layer, the apps'
parameters, the batch's request layout and subscriptions) into device
buffers of static shape and runs the step through the C ABI, in this
order for every layer:

  1. route build (once per step: the batch and subscriptions are shared by
     all hooked layers; when the first layer's first consumer of the routing
     is an SAE encode, or its fused probes + steering pass, that kernel
     builds the routing itself: one launch instead of two);
  2. reads of the activation as the model produced it: per-token probes,
     mean-pooled probes, SAE encodes;
  3. writes: steering, then each SAE app's clamp-decode;
     (by default a layer's per-token probes run fused with its steering,
     after the other reads: one pass reads each row, probes it as read and
     writes the steered row, with the same results as the separate calls);
  4. readback of SAE results into each app's ring (by default fused into
     the encode's merge, which writes the ring rows itself).

Reads before writes means every app at a hook sees the same activation,
whatever else is subscribed.  All buffers are allocated here, once; ``run``
only enqueues kernels, so it can be captured into a HIP graph and replayed
after the device-side inputs (subscriptions, alpha, clamp values) change.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

from . import (XMIX_PROBE_LAST, XMIX_PROBE_MEAN, XMIX_PROBE_TOKEN, Ring, Route, SaeApp, SaeDict,
               probe_workspace, sae_encode_workspace, xmix_probe_score, xmix_readback_compact,
               xmix_route_build, xmix_route_sae_encode_topk_multi, xmix_sae_clamp_decode,
               xmix_sae_clamp_decode_multi, xmix_sae_encode_candidates,
               xmix_sae_encode_topk, xmix_sae_encode_topk_multi, xmix_sae_encode_topk_ring,
               xmix_sae_fold_bias, xmix_route_sae_encode_candidates, xmix_route_steer_probe,
               xmix_sae_merge_topk, xmix_sae_merge_topk_ring, xmix_sae_pack_encoder,
               xmix_steer_apply, xmix_steer_probe)


def to_device_bits(a: np.ndarray, device) -> torch.Tensor:
    """uint16 bf16 bit patterns (numpy) -> torch.bfloat16 on the device."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)


def to_device(a: np.ndarray, dtype, device) -> torch.Tensor:
    if a.dtype == np.uint16:
        return to_device_bits(a, device)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=dtype)


@dataclass
class _Probes:
    mode: int
    w: torch.Tensor
    b: torch.Tensor
    bits: List[int]
    logit: torch.Tensor
    score: torch.Tensor
    ws: Optional[torch.Tensor]


@dataclass
class _Sae:
    bit: int
    m: int
    k: int
    W_enc: SaeDict
    b_enc: torch.Tensor
    b_dec: torch.Tensor
    c_fold: Optional[torch.Tensor]
    idx: torch.Tensor
    val: torch.Tensor
    ws: torch.Tensor
    W_dec: Optional[torch.Tensor] = None
    clamp_ids: Optional[torch.Tensor] = None
    clamp_vals: Optional[torch.Tensor] = None
    ring: Optional[Ring] = None


@dataclass
class _Layer:
    layer_id: int
    h_in: torch.Tensor
    h: torch.Tensor
    steer_v: Optional[torch.Tensor] = None
    steer_bits: List[int] = field(default_factory=list)
    probes: List[_Probes] = field(default_factory=list)
    saes: List[_Sae] = field(default_factory=list)


class HookStep:
    def __init__(self, wl, device="cuda", fold_bias: bool = True, fuse_readback: bool = True,
                 fuse_steer_probe: bool = True, fuse_route: bool = True,
                 batch_saes: bool = True):
        dev = torch.device(device)
        self.wl = wl
        # a layer's SAE apps encoded by one batched call and clamped by
        # another (two launches for every app's candidates and merges, one
        # for every app's clamp) instead of two launches per app and one per
        # clamp; the results are the per-app calls' bit for bit
        self.batch_saes = batch_saes
        self.fuse_readback = fuse_readback
        self.fuse_steer_probe = fuse_steer_probe
        self.fuse_route = fuse_route
        self.device = dev
        act = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.req = to_device(wl.req, torch.int32, dev)
        self.T_valid = torch.tensor([wl.T_valid], dtype=torch.int32, device=dev)
        self.sub = to_device(wl.sub.astype(np.uint32), torch.int32, dev)
        self.alpha = to_device(wl.alpha.astype(np.float32), torch.float32, dev)
        self.err = torch.zeros(1, dtype=torch.int32, device=dev)
        self.cu = None if wl.cu_seqlens is None else to_device(wl.cu_seqlens, torch.int32, dev)
        self.route = Route(wl.T_max, wl.n_apps, dev)
        self.layers: List[_Layer] = []
        for L in wl.layers:
            h_in = to_device(L.h, act, dev)
            lay = _Layer(L.layer_id, h_in, h_in.clone())
            if L.steer:
                lay.steer_v = to_device(np.stack([s.v for s in L.steer]), act, dev)
                lay.steer_bits = [s.bit for s in L.steer]
            for mode, name in ((XMIX_PROBE_TOKEN, "token"), (XMIX_PROBE_MEAN, "mean"),
                               (XMIX_PROBE_LAST, "last")):
                ps = [p for p in L.probes if p.mode == name]
                if not ps:
                    continue
                n_out = wl.T_max if mode == XMIX_PROBE_TOKEN else wl.R_max
                nb = probe_workspace(wl.T_max, len(ps), mode)
                lay.probes.append(_Probes(
                    mode, to_device(np.stack([p.w for p in ps]), act, dev),
                    torch.tensor([p.b for p in ps], dtype=torch.float32, device=dev),
                    [p.bit for p in ps],
                    torch.zeros((len(ps), n_out), dtype=torch.float32, device=dev),
                    torch.zeros((len(ps), n_out), dtype=torch.float32, device=dev),
                    torch.empty(nb, dtype=torch.uint8, device=dev) if nb else None))
            for s in L.saes:
                d = wl.d
                # the dictionary is packed once into the layout the encode streams
                W_row = to_device_bits(s.W_enc, dev)
                W_dict = xmix_sae_pack_encoder(W_row)
                del W_row
                sae = _Sae(
                    s.bit, s.m, s.k, W_dict, to_device_bits(s.b_enc, dev),
                    to_device_bits(s.b_dec, dev), None,
                    torch.zeros((wl.T_max, s.k), dtype=torch.int32, device=dev),
                    torch.zeros((wl.T_max, s.k), dtype=torch.bfloat16, device=dev),
                    torch.empty(sae_encode_workspace(wl.T_max, d, s.m, s.k), dtype=torch.uint8,
                                device=dev))
                if fold_bias:
                    sae.c_fold = torch.empty(s.m, dtype=torch.float32, device=dev)
                    xmix_sae_fold_bias(sae.W_enc, sae.b_enc, sae.b_dec, sae.c_fold)
                if s.W_dec is not None and s.clamp_ids is not None:
                    sae.W_dec = to_device_bits(s.W_dec, dev)
                    sae.clamp_ids = to_device(s.clamp_ids, torch.int32, dev)
                    sae.clamp_vals = to_device(s.clamp_vals, torch.float32, dev)
                if s.ring_capacity:
                    sae.ring = Ring(s.ring_capacity, 16 + s.k * 4 + s.k * 2, dev)
                lay.saes.append(sae)
            self.layers.append(lay)

    def reset(self):
        """Restore every layer's activation to its input value."""
        for lay in self.layers:
            lay.h.copy_(lay.h_in)

    def run(self, stream=None, mark=None, only=None, repeat=1):
        """Enqueue one full hook step (all layers) on `stream`.

        mark: a host callable invoked while enqueueing with the name of each
        stage right before its launch, and with "end" after the last one
        (e.g. to record timing events between the stages); an SAE encode is
        then issued as its two stages ("...encode" and "merge"), which
        enqueues the same kernels.
        only, repeat: enqueue only the stage named `only` (same arguments as
        in the full step; the device state it reads, such as the routing or
        the encode's candidates, is whatever an earlier step left), `repeat`
        times in a row, to time one stage on its own (repeat=0 launches
        nothing)."""
        def issue(name, call):
            if only is not None and name != only:
                return
            if mark is not None:
                mark(name)
            for _ in range(repeat):
                call()

        split = mark is not None or only is not None
        # the kernel that first reads the routing builds it when it can: the
        # first layer's first SAE encode, or its fused probes + steering pass
        # when that is the layer's only read
        first = self.layers[0] if self.layers else None
        # the first layer's token probes, when they run fused with its
        # steering, come after its SAE encodes
        fused_only = first is not None and (not first.probes or (
            self.fuse_steer_probe and first.steer_v is not None and len(first.probes) == 1
            and first.probes[0].mode == XMIX_PROBE_TOKEN))
        route_in_encode = (self.fuse_route and fused_only and len(first.saes) > 0
                           and self.wl.T_max <= 1024)
        route_in_pass = (self.fuse_route and self.fuse_steer_probe and first is not None
                         and not first.saes and first.steer_v is not None
                         and len(first.probes) == 1
                         and first.probes[0].mode == XMIX_PROBE_TOKEN)
        if not (route_in_encode or route_in_pass):
            issue("route", lambda: xmix_route_build(self.req, self.T_valid, self.sub, self.route,
                                                    self.err, stream))
        modes = {XMIX_PROBE_TOKEN: "token", XMIX_PROBE_MEAN: "mean", XMIX_PROBE_LAST: "last"}
        for li, lay in enumerate(self.layers):
            fused = None  # the token probes that run in one pass with the steering
            if self.fuse_steer_probe and lay.steer_v is not None:
                fused = next((p for p in lay.probes if p.mode == XMIX_PROBE_TOKEN), None)
            for p in lay.probes:
                if p is fused:
                    continue
                issue(f"L{li}/probe_{modes[p.mode]}",
                      lambda p=p, lay=lay: xmix_probe_score(
                          lay.h, self.route, p.w, p.b, p.bits, p.mode, p.logit, p.score,
                          cu_seqlens=self.cu, ws=p.ws, stream=stream))
            batched = (self.batch_saes and len(lay.saes) > 1
                       and (self.fuse_readback or all(s.ring is None for s in lay.saes)))
            if batched:
                apps = [SaeApp(s.bit, s.W_enc, s.b_enc, s.b_dec, s.c_fold, s.k, s.idx, s.val,
                               s.ws, s.ring if self.fuse_readback else None, s.bit)
                        for s in lay.saes]
                if route_in_encode and li == 0:
                    issue(f"L{li}/saes/route+encode",
                          lambda lay=lay, apps=apps: xmix_route_sae_encode_topk_multi(
                              self.req, self.T_valid, self.sub, self.route, self.err, lay.h,
                              apps, lay.layer_id, stream))
                else:
                    issue(f"L{li}/saes/encode",
                          lambda lay=lay, apps=apps: xmix_sae_encode_topk_multi(
                              lay.h, self.route, apps, self.req, lay.layer_id, stream))
            for i, s in enumerate(lay.saes if not batched else []):
                routed = route_in_encode and li == 0 and i == 0
                name = f"L{li}/sae{s.bit}"
                if split or routed:
                    if routed:
                        issue(f"{name}/route+encode",
                              lambda s=s, lay=lay: xmix_route_sae_encode_candidates(
                                  self.req, self.T_valid, self.sub, self.route, self.err, lay.h,
                                  s.bit, s.W_enc, s.b_enc, s.b_dec, s.c_fold, s.k, s.ws, stream))
                    else:
                        issue(f"{name}/encode",
                              lambda s=s, lay=lay: xmix_sae_encode_candidates(
                                  lay.h, self.route, s.bit, s.W_enc, s.b_enc, s.b_dec, s.c_fold,
                                  s.k, s.ws, stream))
                    if s.ring is not None and self.fuse_readback:
                        issue(f"{name}/merge",
                              lambda s=s, lay=lay: xmix_sae_merge_topk_ring(
                                  lay.h, self.route, s.bit, s.W_enc, s.c_fold, s.k, s.idx, s.val,
                                  s.ws, self.req, lay.layer_id, s.bit, s.ring, stream))
                    else:
                        issue(f"{name}/merge",
                              lambda s=s, lay=lay: xmix_sae_merge_topk(
                                  lay.h, self.route, s.bit, s.W_enc, s.c_fold, s.k, s.idx, s.val,
                                  s.ws, stream))
                elif s.ring is not None and self.fuse_readback:
                    # the merge writes the ring rows itself
                    issue(name, lambda s=s, lay=lay: xmix_sae_encode_topk_ring(
                        lay.h, self.route, s.bit, s.W_enc, s.b_enc, s.b_dec, s.c_fold, s.k, s.idx,
                        s.val, s.ws, self.req, lay.layer_id, s.bit, s.ring, stream))
                else:
                    issue(name, lambda s=s, lay=lay: xmix_sae_encode_topk(
                        lay.h, self.route, s.bit, s.W_enc, s.b_enc, s.b_dec, s.c_fold, s.k, s.idx,
                        s.val, s.ws, stream))
            if fused is not None and route_in_pass and li == 0:
                issue(f"L{li}/route+steer_probe",
                      lambda lay=lay, fused=fused: xmix_route_steer_probe(
                          self.req, self.T_valid, self.sub, self.route, self.err, lay.h,
                          lay.steer_v, lay.steer_bits, self.alpha, fused.w, fused.b, fused.bits,
                          fused.logit, fused.score, stream))
            elif fused is not None:
                issue(f"L{li}/steer_probe",
                      lambda lay=lay, fused=fused: xmix_steer_probe(
                          lay.h, self.route, self.req, lay.steer_v, lay.steer_bits, self.alpha,
                          fused.w, fused.b, fused.bits, fused.logit, fused.score, stream))
            elif lay.steer_v is not None:
                issue(f"L{li}/steer", lambda lay=lay: xmix_steer_apply(
                    lay.h, self.route, self.req, lay.steer_v, lay.steer_bits, self.alpha, stream))
            clampers = [s for s in lay.saes if s.W_dec is not None]
            if self.batch_saes and len(clampers) > 1:
                issue(f"L{li}/saes/clamp",
                      lambda lay=lay, cs=clampers: xmix_sae_clamp_decode_multi(
                          lay.h, self.route,
                          [(s.bit, s.idx, s.val, s.W_dec, s.clamp_ids, s.clamp_vals) for s in cs],
                          stream))
            else:
                for s in clampers:
                    issue(f"L{li}/sae{s.bit}/clamp",
                          lambda s=s, lay=lay: xmix_sae_clamp_decode(
                              lay.h, self.route, s.bit, s.idx, s.val, s.W_dec, s.clamp_ids,
                              s.clamp_vals, stream=stream))
            for s in lay.saes:
                if s.ring is not None and not self.fuse_readback:
                    issue(f"L{li}/sae{s.bit}/compact",
                          lambda s=s, lay=lay: xmix_readback_compact(
                              [s.idx, s.val], self.route, s.bit, self.req, lay.layer_id, s.bit,
                              s.ring, stream))
        if mark is not None:
            mark("end")

    def stage_names(self):
        """The names of the step's stages, in launch order (as `run` reports
        them to `mark`)."""
        names = []
        self.run(mark=names.append, repeat=0)
        return names[:-1]

    def hbm_bytes(self) -> int:
        """Algorithmic bytes of one step: what the method must touch."""
        wl = self.wl
        esz = 2 if wl.dtype == "bf16" else 4
        sub = wl.sub.astype(np.uint64)
        live = np.zeros(wl.T_max, np.uint64)
        ok = (wl.req >= 0) & (np.arange(wl.T_max) < wl.T_valid)
        live[ok] = sub[wl.req[ok]]
        total = 0
        for L in wl.layers:
            steer_bits = sum(1 << s.bit for s in L.steer)
            read_bits = steer_bits | sum(1 << p.bit for p in L.probes) | sum(1 << s.bit for s in L.saes)
            rows_read = int(np.count_nonzero(live & np.uint64(read_bits)))
            rows_written = int(np.count_nonzero(live & np.uint64(steer_bits | sum(
                1 << s.bit for s in L.saes if s.W_dec is not None))))
            total += (rows_read + rows_written) * wl.d * esz
            total += len(L.steer) * wl.d * esz + len(L.probes) * wl.d * esz
            for s in L.saes:
                total += s.m * wl.d * 2 + s.m * 4        # W_enc + folded bias
                n_sub = int(np.count_nonzero(live & np.uint64(1 << s.bit)))
                total += n_sub * s.k * 6                 # idx + val
                if s.W_dec is not None:
                    total += len(s.clamp_ids) * wl.d * 2
                if s.ring_capacity:
                    total += min(n_sub, s.ring_capacity) * (16 + s.k * 6)
        return total
