"""Hybrid CPU-GPU execution of one MoE layer (SAEM Section IV-D.2).

Host-side driver around the C ABI; all arithmetic happens in the library:

  GPU stream    route + top-k -> repack (packs the offloaded rows) -> grouped FFN
                over the resident and shared experts ------------------> combine
  copy stream          \\-> counts, n_res, offloaded rows to pinned host memory
                                                         \\-> y_off to HBM --/
  host                     (waits for the copy only) -> moe_host_ffn over the
                           offloaded experts, in parallel with the GPU FFN

The device-to-host copy starts as soon as the repack is done, the host runs the
offloaded experts while the GPU streams the resident ones, and the combine
merges both (the merge step of Section IV-D.2).  The copy stream runs at the
default priority, as every stream here does.
"""
from __future__ import annotations

import time
from typing import Callable, Dict, Optional

import numpy as np
import torch

from . import (moe_combine, moe_grouped_ffn, moe_host_ffn, moe_repack, moe_route_topk)


def _np_view(t: torch.Tensor) -> np.ndarray:
    """numpy view of a host tensor (bf16 as uint16 bits), no copy."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class HybridLayer:
    """One layer whose resident experts run on the GPU and offloaded experts on the host.

    dev: a ``device.DeviceLayer`` (HBM copy of the layer, resident experts in slots);
    host_w13(e) / host_w2(e): row-major host weights of expert e ([2F, H] / [H, F],
    the layer dtype), asked for only for experts that have offloaded rows.
    """

    def __init__(self, dev, host_w13: Callable[[int], np.ndarray], host_w2: Callable[[int], np.ndarray],
                 threads: int = 0, pin: bool = True, out_dtype: Optional[int] = None):
        c = dev.cfg
        self.dev = dev
        self.host_w13 = host_w13
        self.host_w2 = host_w2
        self.threads = threads
        self.pin = pin
        T, E, k, H, S = c.tokens, c.experts, c.top_k, c.hidden, c.shared
        self.P = T * k
        self.o = dev.alloc_outputs(out_dtype)
        d = dev.device
        self.y = torch.empty((max(self.P + S * T, 1), H), dtype=torch.float32, device=d)
        self.out = self.o["out"]
        self.d_y_off = torch.empty((max(self.P, 1), H), dtype=torch.float32, device=d)
        self.h_counts = torch.empty((E,), dtype=torch.int32, pin_memory=True)
        self.h_seg = torch.empty((E,), dtype=torch.int32, pin_memory=True)
        self.h_nres = torch.empty((1,), dtype=torch.int32, pin_memory=True)
        self.h_off = torch.empty((max(self.P, 1), H), dtype=dev.tdtype, pin_memory=True)
        self.h_y_off = torch.empty((max(self.P, 1), H), dtype=torch.float32, pin_memory=True)
        self.copy_stream = torch.cuda.Stream(device=d)
        self.ev = {n: torch.cuda.Event(enable_timing=True) for n in
                   ("start", "packed", "d2h", "ffn", "h2d", "end")}
        self._w13: Dict[int, np.ndarray] = {}
        self._w2: Dict[int, np.ndarray] = {}
        self.last: Dict[str, float] = {}

    def _weights(self, e: int):
        if e not in self._w13:
            self._w13[e] = np.ascontiguousarray(self.host_w13(e))
            self._w2[e] = np.ascontiguousarray(self.host_w2(e))
        return self._w13[e], self._w2[e]

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
        moe_repack(dev.dims, o["topk_idx"], o["topk_w"], dev.expert_slot, dev.x, o["counts"], o["seg_start"],
                   o["perm"], o["inv_perm"], o["n_res"], o["off_rows"], o["off_w"], stream=s0)
        ev["packed"].record(s0)
        cs.wait_event(ev["packed"])
        with torch.cuda.stream(cs):
            self.h_counts.copy_(o["counts"], non_blocking=True)
            self.h_seg.copy_(o["seg_start"], non_blocking=True)
            self.h_nres.copy_(o["n_res"], non_blocking=True)
            self.h_off.copy_(o["off_rows"], non_blocking=True)
            ev["d2h"].record(cs)
        moe_grouped_ffn(dev.dims, dev.x, o["perm"], o["counts"], o["seg_start"], dev.expert_slot, dev.w13, dev.w2,
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
        moe_combine(dev.dims, o["topk_idx"], o["topk_w"], o["inv_perm"], dev.expert_slot, self.y,
                    self.d_y_off if n_off > 0 else None, o["n_res"], self.out, o["out_dtype"], stream=s0)
        ev["end"].record(s0)
        self.last = {"n_res": n_res, "n_off": n_off, "host_wait_d2h_ms": (t_d2h - t_launch) * 1e3,
                     "host_ffn_ms": (t_host - t_d2h) * 1e3, "host_t0": t0}
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
        return r
