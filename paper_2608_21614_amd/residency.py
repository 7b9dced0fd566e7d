"""Stage-aware expert residency with real slot copies (SAEM Section IV-C).

Host-side driver of a stack of MoE layers over a stage-structured decode trace;
all arithmetic happens in the library.

* Per layer, a fixed pool of ``n_slots`` expert slots in HBM (Section IV-C.1)
  holds the resident experts' weights in the tile layout; ``expert_slot[l]`` on
  the device is the layer's residency map.
* Every (step, layer) call runs the fused layer forward (``moe_layer_forward``)
  against the current map and adds its per-expert counts to the layer's
  activation log on the device (``moe_stage_accumulate``, Section IV-B.2).
* At a stage boundary the logs come to the host (one small copy), the next
  stage's residency is planned per layer (``moe_stage_plan``: top-N by count,
  incumbents keep their slots, Section IV-C.2), and the incoming experts'
  weights are copied from pinned host memory into the freed slots on a copy
  stream: a row-major host-to-device copy into a staging buffer, then
  ``moe_pack_weights`` into the slot (Section IV-C.3).
* The copies overlap the next stage's first ``lag`` steps.  During those steps
  only the experts that keep their slot are resident (the evicted experts' slots
  are being overwritten, the incoming ones are in flight); before step ``lag``
  of the stage the compute stream waits for the copy event and switches to the
  full map.  ``lag = 0`` switches at once (the wait is then fully exposed).

The copy stream runs at the default priority, as every stream here does.
"""
from __future__ import annotations

from typing import Callable, Dict, List, Optional

import numpy as np
import torch

from . import (MOE_BF16, MOE_F32, layer_args, make_dims, moe_cue_build, moe_cue_step, moe_layer_forward,
               moe_pack_weights, moe_stage_accumulate, moe_stage_plan, moe_workspace_bytes)
from .device import to_device, to_host


class StageResidencyRunner:
    """Runs a ``workloads.StageTrace`` (or any object with the same fields) on one GPU.

    routers[l]: [E, H] router of layer l (host array); host_weights(l, e) -> (w13 [2F, H],
    w2 [H, F]) row-major host arrays of expert e of layer l; x_of(step, l) -> [T, H]
    activations (host array or device tensor).
    """

    def __init__(self, trace, routers: List[np.ndarray], host_weights: Callable[[int, int], tuple],
                 x_of: Callable[[int, int], object], lag: int = 0, device: str = "cuda"):
        c = trace.cfg
        self.trace, self.cfg, self.lag, self.device = trace, c, int(lag), device
        self.host_weights, self.x_of = host_weights, x_of
        L, E, H, F, T, k, N = c.layers, c.experts, c.hidden, c.ffn, c.batch, c.top_k, c.n_slots
        self.dt = MOE_BF16 if c.dtype == "bf16" else MOE_F32
        self.tdtype = torch.bfloat16 if c.dtype == "bf16" else torch.float32
        self.dims = make_dims(T, H, E, F, k, 0, 0, N, self.dt)
        self.ws = torch.empty(moe_workspace_bytes(self.dims), dtype=torch.uint8, device=device)
        self.wr = [to_device(np.asarray(routers[l]), device) for l in range(L)]
        self.bias = to_device(np.asarray(trace.stage_bias, dtype=np.float32), device)    # [stages, L, E]
        self.w13 = [torch.empty((N, 2 * F, H), dtype=self.tdtype, device=device) for _ in range(L)]
        self.w2 = [torch.empty((N, H, F), dtype=self.tdtype, device=device) for _ in range(L)]
        self.st13 = torch.empty((2 * F, H), dtype=self.tdtype, device=device)
        self.st2 = torch.empty((H, F), dtype=self.tdtype, device=device)
        self.log = torch.zeros((L, E), dtype=torch.int64, device=device)
        self.out = torch.empty((T, H), dtype=self.tdtype, device=device)
        self.copy_stream = torch.cuda.Stream(device=device)
        self._pinned: Dict[tuple, tuple] = {}
        self.reset(lag)

    def reset(self, lag: int) -> None:
        """Back to the trace's initial residency (slots refilled, logs cleared); host buffers are kept."""
        c, L, E, dev = self.cfg, self.cfg.layers, self.cfg.experts, self.device
        self.lag = int(lag)
        # initial residency: experts of initial_resident in ascending id take slots 0..N-1
        self.slot = np.full((L, E), -1, dtype=np.int32)
        for l in range(L):
            ids = np.flatnonzero(self.trace.initial_resident[l])
            self.slot[l, ids] = np.arange(len(ids), dtype=np.int32)
        self.d_slot = [to_device(self.slot[l], dev) for l in range(L)]
        self.log.zero_()
        for l in range(L):
            for e in np.flatnonzero(self.slot[l] >= 0):
                self._copy_expert(l, int(e), int(self.slot[l, e]), torch.cuda.current_stream(dev))
        torch.cuda.synchronize(dev)
        self.copies: List[dict] = []      # one record per boundary with copies

    # -- weights --------------------------------------------------------------
    def _host(self, l: int, e: int):
        key = (l, e)
        if key not in self._pinned:
            w13, w2 = self.host_weights(l, e)
            p13 = torch.empty(w13.shape, dtype=self.tdtype, pin_memory=True)
            p2 = torch.empty(w2.shape, dtype=self.tdtype, pin_memory=True)
            for dst, src in ((p13, w13), (p2, w2)):
                src = np.ascontiguousarray(src)
                view = dst.view(torch.int16).numpy().view(np.uint16) if self.tdtype == torch.bfloat16 else dst.numpy()
                view[...] = src
            self._pinned[key] = (p13, p2)
        return self._pinned[key]

    def prepare_host_weights(self, experts_per_layer: Optional[int] = None) -> None:
        """Stage every expert's weights in pinned host memory now (so boundaries only copy)."""
        c = self.cfg
        for l in range(c.layers):
            for e in range(c.experts if experts_per_layer is None else experts_per_layer):
                self._host(l, e)

    def _copy_expert(self, l: int, e: int, s: int, stream) -> None:
        p13, p2 = self._host(l, e)
        with torch.cuda.stream(stream):
            self.st13.copy_(p13, non_blocking=True)
            moe_pack_weights(self.st13, self.w13[l][s], stream=stream)
            self.st2.copy_(p2, non_blocking=True)
            moe_pack_weights(self.st2, self.w2[l][s], stream=stream)

    # -- trace ------------------------------------------------------------------
    def run(self, steps: Optional[int] = None, keep_outputs=(), log_every: int = 0,
            detector: Optional[dict] = None) -> dict:
        """Runs the first `steps` steps.  keep_outputs: (step, layer) pairs whose outputs (and routing) are kept.

        Stage boundaries: without a detector, the trace's own stage ends.  With
        ``detector = {"cues": [...], "stream": [steps, batch] int32}`` they come
        from the cue machine (Section IV-B.1): after every step the batch's
        generated tokens are fed to ``moe_cue_step``, and a cue matched in any
        sequence ends the stage with that step (false positives included).  The
        router bias still follows the trace's true stages.
        """
        c, tr = self.cfg, self.trace
        L, E, T, k = c.layers, c.experts, c.batch, c.top_k
        steps = c.steps if steps is None else int(steps)
        main = torch.cuda.current_stream(self.device)
        stage_of = tr.stage_of_step()
        ends = set(int(v) for v in tr.stage_ends()[:-1])
        if detector is not None:
            fsm = moe_cue_build(detector["cues"])
            tokens = np.ascontiguousarray(detector["stream"], dtype=np.int32)
            cue_state = np.zeros(tokens.shape[1], dtype=np.int32)
        boundary_steps = []
        counts = torch.empty((steps, L, E), dtype=torch.int32, device=self.device)
        n_res = torch.empty((steps, L), dtype=torch.int32, device=self.device)
        kept = {}
        kept_idx = {}
        keep = set(keep_outputs)
        used_slot = np.empty((steps, L, E), dtype=np.int32)  # map each call ran with
        cur = self.slot.copy()          # map on the device now
        pending = None                  # (switch_step, final map, copy event)
        hist = [self.slot.copy()]
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        stalls = []
        ev0.record(main)

        def set_maps(new_map, d_maps):
            # stream-ordered device copies of maps uploaded at the boundary (no host wait)
            nonlocal cur
            for l in range(L):
                if not np.array_equal(new_map[l], cur[l]):
                    self.d_slot[l].copy_(d_maps[l], non_blocking=True)
            cur = new_map.copy()

        def finish_pending():
            nonlocal pending
            sw, final, d_final, ev_copy = pending
            e_a = torch.cuda.Event(enable_timing=True)
            e_b = torch.cuda.Event(enable_timing=True)
            e_a.record(main)
            main.wait_event(ev_copy)
            e_b.record(main)
            stalls.append((e_a, e_b))
            set_maps(final, d_final)
            pending = None

        for step in range(steps):
            if pending is not None and step >= pending[0]:
                finish_pending()
            s = int(stage_of[step])
            for l in range(L):
                x = self.x_of(step, l)
                if not isinstance(x, torch.Tensor):
                    x = to_device(np.asarray(x), self.device)
                kept_call = (step, l) in keep
                out = torch.empty_like(self.out) if kept_call else self.out
                idx = torch.empty((T, k), dtype=torch.int32, device=self.device) if kept_call else None
                args = layer_args(self.dims, x, self.wr[l], self.bias[s, l], self.d_slot[l], self.w13[l], self.w2[l],
                                  None, None, out, self.dt, topk_idx=idx, counts=counts[step, l],
                                  n_res=n_res[step, l:l + 1])
                moe_layer_forward(args, self.ws, main)
                moe_stage_accumulate(E, counts[step, l], self.log[l], main)
                if kept_call:
                    kept[(step, l)] = out
                    kept_idx[(step, l)] = idx
            used_slot[step] = cur
            if detector is not None:
                boundary = bool((moe_cue_step(fsm, tokens[step], cue_state) >= 0).any())
            else:
                boundary = step in ends
            if boundary and step + 1 < steps:
                boundary_steps.append(step)
                if pending is not None:   # a stage shorter than the lag: its copies must land first
                    finish_pending()
                h_log = to_host(self.log)                        # waits for this stage's calls
                new = np.stack([moe_stage_plan(h_log[l], cur[l], c.n_slots) for l in range(L)])
                self.log.zero_()
                stay = np.where((new >= 0) & (new == cur), new, -1).astype(np.int32)
                incoming = [(l, int(e), int(new[l, e])) for l in range(L) for e in range(E)
                            if new[l, e] >= 0 and cur[l, e] != new[l, e]]
                hist.append(new.copy())
                d_new = to_device(new, self.device)              # [L, E]; the host already waited above
                if incoming:
                    # evicted and incoming experts leave the map before their slots are overwritten
                    set_maps(stay, to_device(stay, self.device))
                    ev_b = torch.cuda.Event()
                    ev_b.record(main)
                    cs = self.copy_stream
                    cs.wait_event(ev_b)
                    rec = {"step": step, "experts": len(incoming), "start": torch.cuda.Event(enable_timing=True),
                           "end": torch.cuda.Event(enable_timing=True)}
                    rec["start"].record(cs)
                    for l, e, sl in incoming:
                        self._copy_expert(l, e, sl, cs)
                    rec["end"].record(cs)
                    self.copies.append(rec)
                    pending = (step + 1 + self.lag, new.copy(), d_new, rec["end"])
                    if self.lag == 0:
                        finish_pending()
                else:
                    set_maps(new, d_new)
            if log_every and step % log_every == 0:
                print(f"[residency] step {step}/{steps} stage {s}", flush=True)
        if pending is not None:
            finish_pending()
        ev1.record(main)
        torch.cuda.synchronize(self.device)
        self.slot = cur.copy()
        cnt = to_host(counts).astype(np.int64)
        nr = to_host(n_res).astype(np.int64)
        b = 2 if self.tdtype == torch.bfloat16 else 4
        expert_bytes = 3 * c.hidden * c.ffn * b
        copy_ms = [r["start"].elapsed_time(r["end"]) for r in self.copies]
        n_copied = sum(r["experts"] for r in self.copies)
        total = int(cnt.sum())
        return {
            "counts": cnt, "n_res": nr, "used_slot": used_slot, "slot_history": np.stack(hist),
            "outputs": kept, "topk_idx": {key: to_host(v) for key, v in kept_idx.items()},
            "chr_online": float(nr.sum()) / total if total else 1.0,
            "trace_ms": ev0.elapsed_time(ev1), "calls": steps * L,
            "copied_experts": n_copied, "copy_ms_total": float(sum(copy_ms)),
            "copy_GBps": (n_copied * expert_bytes / (sum(copy_ms) * 1e-3) / 1e9) if copy_ms else None,
            "stall_ms_total": float(sum(a.elapsed_time(b_) for a, b_ in stalls)),
            "boundaries_with_copies": len(self.copies), "lag": self.lag,
            "boundary_steps": np.asarray(boundary_steps, dtype=np.int64),
        }
