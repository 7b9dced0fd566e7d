"""Bookkeeping baseline of one MoE layer: per-expert mask, gather, FFN launch, scatter-add.

The in-house A/B for expert-aligned repacking (SAEM Section III, Fig. of the
decode-time breakdown, and Section IV-E.1): the same router and FFN kernels as
the fused path, driven the way a framework without repacking drives them.  For
every resident expert the host finds its (token, choice) pairs with a mask and
a nonzero (which waits for the device), gathers the rows, launches the expert's
FFN on them alone, and adds the weighted result back into the output with an
atomic scatter-add.  Shared experts run once over all tokens.

Only the bookkeeping (masks, nonzero, gathers, the scatter-add) uses PyTorch
operators, because it is the baseline's own structure; the expert FFN is the
library's kernel in both paths.  Offloaded experts are the host path's in both
(not computed here), so the output is the resident partial sum, as the fused
path's is without ``y_off``.
"""
from __future__ import annotations

import time
from typing import Dict

import torch

from . import make_dims, moe_grouped_ffn, moe_route_topk, moe_workspace_bytes


class BookkeepingLayer:
    def __init__(self, dev):
        c = dev.cfg
        self.dev, self.cfg = dev, c
        T, E, k, H = c.tokens, c.experts, c.top_k, c.hidden
        d = dev.device
        self.o = dev.alloc_outputs()
        self.out = torch.empty((T, H), dtype=torch.float32, device=d)
        self.rows_y = torch.empty((T, H), dtype=torch.float32, device=d)
        self.iota = torch.arange(T, dtype=torch.int32, device=d)        # perm of a one-expert call
        self.count_of = torch.arange(T + 1, dtype=torch.int32, device=d)  # count_of[c] = c
        self.zero = torch.zeros(1, dtype=torch.int32, device=d)
        self.slot_of = dev.layer.expert_slot
        self.resident = [e for e in range(E) if 0 <= int(self.slot_of[e]) < dev.slots]
        ws = max(moe_workspace_bytes(self._dims(n)) for n in range(1, T + 1))
        if c.shared:
            ws = max(ws, moe_workspace_bytes(self._dims(T, shared=True)))
        self.ws = torch.empty(ws, dtype=torch.uint8, device=d)
        self.last: Dict[str, float] = {}

    def _dims(self, rows: int, shared: bool = False):
        c = self.cfg
        F = c.shared_ffn if shared else c.ffn
        return make_dims(rows, c.hidden, 1, F, 1, 0, 0, 1, self.dev.dtype_code)

    def _expert(self, rows_x, n: int, w13, w2, shared: bool = False) -> torch.Tensor:
        """The library's FFN on n gathered rows for one expert (one slot's weights)."""
        y = self.rows_y[:n]
        moe_grouped_ffn(self._dims(n, shared), rows_x, self.iota[:n], self.count_of[n:n + 1], self.zero, self.zero,
                        w13, w2, None, None, y, self.ws)
        return y

    def forward(self) -> torch.Tensor:
        dev, o, c = self.dev, self.o, self.cfg
        t0 = time.perf_counter()
        moe_route_topk(dev.dims, dev.x, dev.w_router, dev.bias, o["logits"], o["topk_idx"], o["topk_w"], dev.ws)
        self.out.zero_()
        idx, w = o["topk_idx"], o["topk_w"]
        syncs = 0
        for e in self.resident:
            pos = (idx == e).nonzero()                      # waits for the device: the count is needed on the host
            syncs += 1
            n = int(pos.shape[0])
            if n == 0:
                continue
            tok, j = pos[:, 0], pos[:, 1]
            rows = dev.x.index_select(0, tok)
            gate = w[tok, j]
            s = int(self.slot_of[e])
            y = self._expert(rows, n, dev.w13[s:s + 1], dev.w2[s:s + 1])
            self.out.index_add_(0, tok, y * gate[:, None])
        for s in range(c.shared):
            y = self._expert(dev.x, c.tokens, dev.ws13[s:s + 1], dev.ws2[s:s + 1], shared=True)
            self.out.add_(y)
        self.last = {"host_syncs": syncs, "host_ms": (time.perf_counter() - t0) * 1e3}
        return self.out
