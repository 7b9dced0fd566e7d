"""Hybrid CPU-GPU execution of one MoE layer (SAEM Section IV-D).

Host-side driver around the C ABI; all arithmetic happens in the library:

  GPU stream    route + top-k -> repack (packs the offloaded rows) -> grouped FFN
                over the resident and shared experts ------------------> combine
  copy stream          \\-> counts, n_res, offloaded rows to pinned host memory
                                                         \\-> y_off to HBM --/
  host                     (waits for the copy only) -> moe_host_ffn over the
                           offloaded experts, in parallel with the GPU FFN

The device-to-host copy starts as soon as the repack is done, the host runs the
offloaded experts while the GPU streams the resident ones, and the combine
merges both (the merge step of Section IV-D.2).

With a cost model (``rates``, Section IV-D.1) and temporary slots, the host
first decides per offloaded expert whether copying it to the GPU beats running
it on the host (``moe_offload_plan``: few tokens favour the host, many the
copy, while the link's queue stays shorter than the host's).  The batch is
repacked with the chosen experts resident and the new offloaded list shipped to
the host; meanwhile a second copy stream moves the chosen experts' weights from
pinned host memory into temporary slots (staging + ``moe_pack_weights``), the
GPU FFN waits for them, and the remaining offloaded experts run on the host as
above.  Every stream runs at the default priority.
"""
from __future__ import annotations

import time
from typing import Callable, Dict, Optional

import numpy as np
import torch

from . import (moe_combine, moe_grouped_ffn, moe_host_ffn, moe_offload_plan, moe_pack_weights, moe_repack,
               moe_route_topk)
from .device import to_device


def _np_view(t: torch.Tensor) -> np.ndarray:
    """numpy view of a host tensor (bf16 as uint16 bits), no copy."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class HybridLayer:
    """One layer whose resident experts run on the GPU and offloaded experts on the host.

    dev: a ``device.DeviceLayer`` (HBM copy of the layer, resident experts in slots).
    Slots of dev beyond those its residency map uses serve as temporary slots for
    experts the cost model copies in (build dev with ``n_slots`` = resident + spare).
    host_w13(e) / host_w2(e): row-major host weights of expert e ([2F, H] / [H, F],
    the layer dtype), asked for only for experts that are offloaded.
    rates: a ``moe_offload_rates`` (None: every offloaded expert runs on the host).
    """

    def __init__(self, dev, host_w13: Callable[[int], np.ndarray], host_w2: Callable[[int], np.ndarray],
                 threads: int = 0, pin: bool = True, out_dtype: Optional[int] = None, rates=None):
        c = dev.cfg
        self.dev = dev
        self.host_w13 = host_w13
        self.host_w2 = host_w2
        self.threads = threads
        self.pin = pin
        self.rates = rates
        T, E, k, H, S, F = c.tokens, c.experts, c.top_k, c.hidden, c.shared, c.ffn
        self.P = T * k
        self.o = dev.alloc_outputs(out_dtype)
        d = dev.device
        self.base_map = np.asarray(dev.layer.expert_slot, dtype=np.int32).copy()
        used = set(int(s) for s in self.base_map if 0 <= s < dev.slots)
        self.tmp_slots = [s for s in range(dev.slots) if s not in used]
        self.d_map = dev.expert_slot                   # map of the call (base, or with temporary slots)
        self.y = torch.empty((max(self.P + S * T, 1), H), dtype=torch.float32, device=d)
        self.out = self.o["out"]
        self.d_y_off = torch.empty((max(self.P, 1), H), dtype=torch.float32, device=d)
        self.h_counts = torch.empty((E,), dtype=torch.int32, pin_memory=True)
        self.h_seg = torch.empty((E,), dtype=torch.int32, pin_memory=True)
        self.h_nres = torch.empty((1,), dtype=torch.int32, pin_memory=True)
        self.h_off = torch.empty((max(self.P, 1), H), dtype=dev.tdtype, pin_memory=True)
        self.h_y_off = torch.empty((max(self.P, 1), H), dtype=torch.float32, pin_memory=True)
        if self.rates is not None and self.tmp_slots:
            self.st13 = torch.empty((2 * F, H), dtype=dev.tdtype, device=d)
            self.st2 = torch.empty((H, F), dtype=dev.tdtype, device=d)
        self.copy_stream = torch.cuda.Stream(device=d)      # offloaded list out, y_off in
        self.weight_stream = torch.cuda.Stream(device=d)    # expert weights in (cost-model copies)
        self.ev = {n: torch.cuda.Event(enable_timing=True) for n in
                   ("start", "packed", "d2h", "copies0", "copies1", "ffn", "h2d", "end")}
        self._w: Dict[int, tuple] = {}
        self._pinned: Dict[int, tuple] = {}
        self.last: Dict[str, float] = {}

    def _weights(self, e: int):
        if e not in self._w:
            self._w[e] = (np.ascontiguousarray(self.host_w13(e)), np.ascontiguousarray(self.host_w2(e)))
        return self._w[e]

    def _pinned_weights(self, e: int):
        if e not in self._pinned:
            pair = []
            for a in self._weights(e):
                t = torch.empty(a.shape, dtype=self.dev.tdtype, pin_memory=True)
                _np_view(t)[...] = a
                pair.append(t)
            self._pinned[e] = tuple(pair)
        return self._pinned[e]

    def _repack_and_ship(self, expert_slot, s0, cs):
        """Repack against `expert_slot`, then copy counts, n_res and offloaded rows to the host."""
        dev, o, ev = self.dev, self.o, self.ev
        moe_repack(dev.dims, o["topk_idx"], o["topk_w"], expert_slot, dev.x, o["counts"], o["seg_start"],
                   o["perm"], o["inv_perm"], o["n_res"], o["off_rows"], o["off_w"], stream=s0)
        ev["packed"].record(s0)
        cs.wait_event(ev["packed"])
        with torch.cuda.stream(cs):
            self.h_counts.copy_(o["counts"], non_blocking=True)
            self.h_seg.copy_(o["seg_start"], non_blocking=True)
            self.h_nres.copy_(o["n_res"], non_blocking=True)
            self.h_off.copy_(o["off_rows"], non_blocking=True)
            ev["d2h"].record(cs)

    def forward(self) -> torch.Tensor:
        """Full layer output [T, H] (resident + shared + offloaded experts); returns self.out."""
        dev, o, ev = self.dev, self.o, self.ev
        c = dev.cfg
        s0 = torch.cuda.current_stream(dev.device)
        cs = self.copy_stream
        E, P = c.experts, self.P
        t0 = time.perf_counter()
        ev["start"].record(s0)
        moe_route_topk(dev.dims, dev.x, dev.w_router, dev.bias, o["logits"], o["topk_idx"], o["topk_w"], dev.ws,
                       stream=s0)
        self._repack_and_ship(dev.expert_slot, s0, cs)
        copied = []
        expert_slot = dev.expert_slot
        if self.rates is not None and self.tmp_slots:
            ev["d2h"].synchronize()
            choice = moe_offload_plan(self.h_counts.numpy(), self.base_map, dev.slots, self.rates,
                                      len(self.tmp_slots))
            copied = [int(e) for e in np.flatnonzero(choice == 1)]
            if copied:
                new_map = self.base_map.copy()
                for e, s in zip(copied, self.tmp_slots):
                    new_map[e] = s
                expert_slot = to_device(new_map, dev.device)
                # the new offloaded list goes out first, on its own stream, so the host
                # never waits behind the weight copies
                self._repack_and_ship(expert_slot, s0, cs)
                ws_ = self.weight_stream
                ws_.wait_event(ev["packed"])      # slots of the previous call are no longer read
                ev["copies0"].record(ws_)
                with torch.cuda.stream(ws_):
                    for e, s in zip(copied, self.tmp_slots):
                        p13, p2 = self._pinned_weights(e)
                        self.st13.copy_(p13, non_blocking=True)
                        moe_pack_weights(self.st13, dev.w13[s], stream=ws_)
                        self.st2.copy_(p2, non_blocking=True)
                        moe_pack_weights(self.st2, dev.w2[s], stream=ws_)
                ev["copies1"].record(ws_)
                s0.wait_event(ev["copies1"])
        moe_grouped_ffn(dev.dims, dev.x, o["perm"], o["counts"], o["seg_start"], expert_slot, dev.w13, dev.w2,
                        dev.ws13, dev.ws2, self.y, dev.ws, stream=s0)
        ev["ffn"].record(s0)
        t_launch = time.perf_counter()
        ev["d2h"].synchronize()
        t_d2h = time.perf_counter()
        n_res = int(self.h_nres[0])
        n_off = P - n_res
        counts = self.h_counts.numpy()
        seg = self.h_seg.numpy()
        if n_off > 0:
            w13 = [None] * E
            w2 = [None] * E
            for e in range(E):
                if counts[e] > 0 and seg[e] >= n_res:
                    w13[e], w2[e] = self._weights(e)
            moe_host_ffn(dev.dims, counts, seg, n_res, w13, w2, _np_view(self.h_off)[:n_off],
                         y_off=self.h_y_off.numpy()[:n_off], threads=self.threads, pin=self.pin)
        t_host = time.perf_counter()
        with torch.cuda.stream(cs):
            if n_off > 0:
                self.d_y_off[:n_off].copy_(self.h_y_off[:n_off], non_blocking=True)
            ev["h2d"].record(cs)
        s0.wait_event(ev["h2d"])
        moe_combine(dev.dims, o["topk_idx"], o["topk_w"], o["inv_perm"], expert_slot, self.y,
                    self.d_y_off if n_off > 0 else None, o["n_res"], self.out, o["out_dtype"], stream=s0)
        ev["end"].record(s0)
        self.d_map = expert_slot
        self.last = {"n_res": n_res, "n_off": n_off, "copied_experts": len(copied),
                     "host_wait_d2h_ms": (t_d2h - t_launch) * 1e3, "host_ffn_ms": (t_host - t_d2h) * 1e3,
                     "host_t0": t0}
        return self.out

    def timings(self) -> Dict[str, float]:
        """Times of the last forward (ms); call after synchronising."""
        ev = self.ev
        r = dict(self.last)
        r["gpu_route_repack_ms"] = ev["start"].elapsed_time(ev["packed"])
        r["gpu_ffn_done_ms"] = ev["start"].elapsed_time(ev["ffn"])
        r["offload_list_on_host_ms"] = ev["start"].elapsed_time(ev["d2h"])
        r["y_off_on_device_ms"] = ev["start"].elapsed_time(ev["h2d"])
        r["layer_ms"] = ev["start"].elapsed_time(ev["end"])
        if r["copied_experts"]:
            r["copy_ms"] = ev["copies0"].elapsed_time(ev["copies1"])
        return r
