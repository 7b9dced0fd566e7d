"""Device-side buffers of one synthetic MoE layer and a fused-forward runner.

Plumbing only: uploads the seeded host tensors of a ``workloads.SyntheticLayer``
to HBM as torch tensors, packs each resident expert's weights into its slot in
the tile layout (``moe_pack_weights``), allocates the outputs and the workspace
once, and calls ``moe_layer_forward``.  No arithmetic of the layer happens here.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from . import (MOE_BF16, MOE_F32, MOE_LOGITS_IN, layer_args, make_dims, moe_layer_forward, moe_pack_weights,
               moe_workspace_bytes)


def to_device(a: np.ndarray, device="cuda") -> torch.Tensor:
    """numpy (uint16 bf16 bits / float32 / int32 / int64) -> device tensor of the matching torch dtype."""
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def to_host(t: torch.Tensor) -> np.ndarray:
    """device tensor -> numpy (bf16 comes back as uint16 bits)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class DeviceLayer:
    """HBM copy of one layer: activations, router, slot-major expert weights, shared experts."""

    def __init__(self, layer, device="cuda", slot_experts: Optional[np.ndarray] = None, n_slots: Optional[int] = None):
        c = layer.cfg
        self.layer = layer
        self.cfg = c
        self.device = device
        self.dtype_code = MOE_BF16 if c.dtype == "bf16" else MOE_F32
        self.tdtype = torch.bfloat16 if c.dtype == "bf16" else torch.float32
        self.x = to_device(layer.x, device)
        self.w_router = to_device(layer.w_router, device)
        self.bias = None if layer.bias is None else to_device(layer.bias, device)
        self.expert_slot = to_device(layer.expert_slot, device)
        se = layer.slot_experts() if slot_experts is None else np.asarray(slot_experts)
        self.slots = int(len(se)) if n_slots is None else int(n_slots)
        H, F = c.hidden, c.ffn
        self.w13 = torch.empty((max(self.slots, 1), 2 * F, H), dtype=self.tdtype, device=device)
        self.w2 = torch.empty((max(self.slots, 1), H, F), dtype=self.tdtype, device=device)
        for s, e in enumerate(se):
            moe_pack_weights(to_device(layer.w13(int(e)), device), self.w13[s])
            moe_pack_weights(to_device(layer.w2(int(e)), device), self.w2[s])
        if c.shared > 0:
            Fs = c.shared_ffn
            self.ws13 = torch.empty((c.shared, 2 * Fs, H), dtype=self.tdtype, device=device)
            self.ws2 = torch.empty((c.shared, H, Fs), dtype=self.tdtype, device=device)
            for s in range(c.shared):
                moe_pack_weights(to_device(layer.ws13(s), device), self.ws13[s])
                moe_pack_weights(to_device(layer.ws2(s), device), self.ws2[s])
        else:
            self.ws13 = self.ws2 = None
        self.dims = make_dims(c.tokens, c.hidden, c.experts, c.ffn, c.top_k, c.shared, c.shared_ffn if c.shared else 0,
                              self.slots, self.dtype_code)
        self.ws = torch.empty(moe_workspace_bytes(self.dims), dtype=torch.uint8, device=device)

    def set_residency(self, expert_slot: np.ndarray) -> None:
        self.expert_slot.copy_(to_device(np.asarray(expert_slot, dtype=np.int32), self.device))

    def alloc_outputs(self, out_dtype: Optional[int] = None) -> Dict[str, torch.Tensor]:
        c = self.cfg
        T, E, k, H = c.tokens, c.experts, c.top_k, c.hidden
        od = self.dtype_code if out_dtype is None else out_dtype
        dev = self.device
        return {
            "out": torch.empty((T, H), dtype=torch.bfloat16 if od == MOE_BF16 else torch.float32, device=dev),
            "out_dtype": od,
            "logits": torch.empty((T, E), dtype=torch.float32, device=dev),
            "topk_idx": torch.empty((T, k), dtype=torch.int32, device=dev),
            "topk_w": torch.empty((T, k), dtype=torch.float32, device=dev),
            "counts": torch.empty((E,), dtype=torch.int32, device=dev),
            "seg_start": torch.empty((E,), dtype=torch.int32, device=dev),
            "perm": torch.empty((max(T * k, 1),), dtype=torch.int32, device=dev),
            "inv_perm": torch.empty((max(T * k, 1),), dtype=torch.int32, device=dev),
            "n_res": torch.empty((1,), dtype=torch.int32, device=dev),
            "off_rows": torch.empty((max(T * k, 1), H), dtype=self.tdtype, device=dev),
            "off_w": torch.empty((max(T * k, 1),), dtype=torch.float32, device=dev),
        }

    def args(self, o: Dict[str, torch.Tensor], logits_in: bool = False, x: Optional[torch.Tensor] = None,
             keep_intermediates: bool = True, pack_offloaded: bool = True):
        """moe_layer_args over this layer and the output buffers in ``o``.

        pack_offloaded=False leaves the offloaded-row list out (no pack), as an expert-parallel
        shard does: the rows of experts it does not hold are another GPU's work, not the host's.
        """
        kw = {}
        if keep_intermediates:
            names = ("topk_idx", "topk_w", "counts", "seg_start", "perm", "inv_perm", "n_res")
            kw = {n: o[n] for n in names + (("off_rows", "off_w") if pack_offloaded else ())}
        return layer_args(self.dims, self.x if x is None else x, self.w_router, self.bias, self.expert_slot,
                          self.w13, self.w2, self.ws13, self.ws2, o["out"], o["out_dtype"],
                          MOE_LOGITS_IN if logits_in else 0, logits=o["logits"], **kw)

    def forward(self, o: Dict[str, torch.Tensor], logits_in: bool = False, stream=None) -> None:
        args = self.args(o, logits_in)
        moe_layer_forward(args, self.ws, stream)
