"""Stage-structured decode trace on the device (SAEM Sections IV-B.2 and IV-C.2).

Host-side driver of the stage-aware residency loop around the layer kernels:
for every decode step and every stacked layer it routes and repacks the batch
through the C ABI (``moe_route_topk``, ``moe_repack``) against that layer's
current residency map, and adds the call's per-expert counts into the layer's
device activation log (``moe_stage_accumulate``).  At the end of each stage it
copies the logs to the host (one small copy), plans the next stage's residency
per layer (``moe_stage_plan``: top-N by the completed stage's counts, fixed
slots), updates the residency maps, and clears the logs.

Routing does not depend on where the experts live, so this loop is the whole
residency trajectory of the trace; the expert FFN of a call runs with the same
maps through ``moe_layer_forward``.  Slot refreshes here update the maps only;
copying expert weights into refreshed slots is outside this loop.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (MOE_BF16, make_dims, moe_repack, moe_route_topk, moe_stage_accumulate, moe_stage_plan,
               moe_workspace_bytes)
from .device import to_device, to_host


def run_routing_trace(trace, routers, device="cuda", log_every: int = 0, x_of=None):
    """Replays ``trace`` (a ``workloads.StageTrace``) with per-layer router weights ``routers[l]``.

    x_of(step, layer) -> [T, H] activations (default: ``trace.x``).

    Returns numpy arrays: counts [steps, layers, E], n_res [steps, layers],
    topk_idx [steps, layers, T, k], slot_history [n_stages, layers, E], and the
    online cache-hit ratio (resident pairs / all pairs).
    """
    c = trace.cfg
    L, E, T, k, H = c.layers, c.experts, c.batch, c.top_k, c.hidden
    dims = make_dims(T, H, E, c.ffn, k, slots=c.n_slots, dtype=MOE_BF16)
    ws = torch.empty(moe_workspace_bytes(dims), dtype=torch.uint8, device=device)
    wr = [to_device(routers[l], device) for l in range(L)]
    bias = to_device(trace.stage_bias, device)                     # [stages, L, E]
    slot = np.stack([np.where(trace.initial_resident[l], 0, -1).astype(np.int32) for l in range(L)])
    for l in range(L):                                              # slots 0..n-1 in expert order
        ids = np.flatnonzero(trace.initial_resident[l])
        slot[l, ids] = np.arange(len(ids), dtype=np.int32)
    d_slot = [to_device(slot[l], device) for l in range(L)]
    log = torch.zeros((L, E), dtype=torch.int64, device=device)
    counts = torch.empty((c.steps, L, E), dtype=torch.int32, device=device)
    n_res = torch.empty((c.steps, L), dtype=torch.int32, device=device)
    idx = torch.empty((c.steps, L, T, k), dtype=torch.int32, device=device)
    w = torch.empty((T, k), dtype=torch.float32, device=device)
    logits = torch.empty((T, E), dtype=torch.float32, device=device)
    seg = torch.empty(E, dtype=torch.int32, device=device)
    perm = torch.empty(T * k, dtype=torch.int32, device=device)
    inv = torch.empty(T * k, dtype=torch.int32, device=device)
    stage_of = trace.stage_of_step()
    ends = set(int(e) for e in trace.stage_ends())
    hist = np.empty((trace.n_stages, L, E), dtype=np.int32)
    hist[0] = slot
    for step in range(c.steps):
        s = int(stage_of[step])
        for l in range(L):
            x = to_device((x_of or trace.x)(step, l), device)
            moe_route_topk(dims, x, wr[l], bias[s, l], logits, idx[step, l], w, ws)
            moe_repack(dims, idx[step, l], w, d_slot[l], None, counts[step, l], seg, perm, inv, n_res[step, l:l + 1])
            moe_stage_accumulate(E, counts[step, l], log[l])
        if step in ends and s + 1 < trace.n_stages:
            h_log = to_host(log)                                   # synchronises the stream
            for l in range(L):
                slot[l] = moe_stage_plan(h_log[l], slot[l], c.n_slots)
                d_slot[l].copy_(to_device(slot[l], device))
            log.zero_()
            hist[s + 1] = slot
        if log_every and step % log_every == 0:
            print(f"[trace] step {step}/{c.steps} stage {s}", flush=True)
    torch.cuda.synchronize()
    cnt = to_host(counts)
    nr = to_host(n_res)
    total = int(cnt.sum())
    return {"counts": cnt, "n_res": nr, "topk_idx": to_host(idx), "slot_history": hist,
            "chr_online": float(nr.sum()) / total if total else 1.0}


def temporal_coherence(counts: np.ndarray, stage_len: np.ndarray) -> float:
    """Sequence-level temporal coherence TC_seq of a routed trace (Section III, Motivation 2).

    counts[step, layer, e]: routed pairs per expert of every (step, layer) call.
    A stage's activation matrix has one row per layer: the fraction of the
    layer's routed tokens that went to each expert over the stage.  TC_seq is
    the mean, over consecutive stages, of the layer-averaged cosine similarity
    of their rows (cosines do not depend on how each row is normalised, so the
    per-stage counts serve directly).  NaN for a trace of one stage.
    """
    c = np.asarray(counts, dtype=np.float64)
    ends = np.cumsum(np.asarray(stage_len, dtype=np.int64))
    starts = ends - np.asarray(stage_len, dtype=np.int64)
    if len(ends) < 2:
        return float("nan")
    R = np.stack([c[a:b].sum(axis=0) for a, b in zip(starts, ends)])     # [P, L, E]
    norm = np.linalg.norm(R, axis=2)                                     # [P, L]
    cos = (R[:-1] * R[1:]).sum(axis=2) / (norm[:-1] * norm[1:])          # [P-1, L]
    return float(cos.mean(axis=1).mean())


def clairvoyant_chr(counts: np.ndarray, stage_len: np.ndarray, n_slots: int) -> float:
    """Cache-hit ratio of the prediction oracle of Section V-C: every stage runs with
    the residency planned from its own activation log (its n_slots most used experts
    per layer, ties to the lower id), the upper bound of the online policy."""
    c = np.asarray(counts, dtype=np.int64)
    ends = np.cumsum(np.asarray(stage_len, dtype=np.int64))
    starts = ends - np.asarray(stage_len, dtype=np.int64)
    total = int(c.sum())
    if total == 0:
        return 1.0
    hits = 0
    for a, b in zip(starts, ends):
        log = c[a:b].sum(axis=0)                                    # [L, E]
        for row in log:
            order = np.lexsort((np.arange(row.size), -row))        # count descending, then id ascending
            hits += int(row[order[:n_slots]].sum())
    return hits / total
