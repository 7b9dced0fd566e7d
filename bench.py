#!/usr/bin/env python
"""MoE-layer forward throughput on one MI355X.

One step = one fused ``moe_layer_forward`` call on one decode batch: router
scores + top-k gate, expert-aligned repacking with the residency split, the
pack of the offloaded rows, the grouped SwiGLU FFN over the resident experts
(two kernels), and the deterministic combine.  The inputs are resident in HBM
before timing starts; each step uses the next of ``--copies`` copies of the
expert weights so that no step finds the previous step's weights in the
256 MB last-level cache.

Prints one JSON line on stdout:
* value: tokens per second of the whole layer forward;
* roofline: the dominant kernel (FFN phase 1: gate/up projections + SwiGLU),
  its algorithmic bytes per launch / its mean duration from HIP events recorded
  by the library around that kernel on the launch stream, against 8 TB/s (decode
  batches); for prefill-size batches (more than 64 tokens) its algorithmic
  FLOPs per launch / the same duration, against 2.5 PFLOP/s dense bf16;
* cpu_baseline: the CPU oracle timed on this host on the same workload;
* workloads: the same measurement (step time, tokens/s, dominant-kernel and
  whole-layer rooflines, stage breakdown, a shorter CPU-oracle sample) for every
  other config -- the tiny fp32 layer, the shared+routed decode batch, the
  prefill chunk (MFMA utilisation), one layer call of the stage-structured
  trace and the Qwen3-MoE-like decode batch -- unless --only is given;
* ep_shards (per workload, unless --ep 0): each GPU's share of the layer under
  8-way expert parallelism timed as its own call on this GPU, beside the layer
  with every expert resident on one GPU (the cross-GPU sum is not built).
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, 8 TB/s
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16
MFMA_F32_PEAK_TFLOPS = 157.3    # dense fp32
METRIC = "MoE-layer tokens/sec + achieved HBM GB/s (expert weights) at decode batch"
TRAFFIC_DIR = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2608_21614_amd", "csrc", n) for n in ("ffn.hip", "common.hpp")]
STAGES = ["route_topk", "repack", "offload_pack", "ffn_phase1", "ffn_phase2", "combine"]
EVENT_EVERY = 4  # timed steps per step that records the dominant kernel's events


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(workload: str):
    """HBM bytes per launch of the dominant kernel from committed counter runs, or None if stale/missing."""
    path = os.path.join(TRAFFIC_DIR, f"traffic_ffn_phase1_{workload}.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        m = re.match(r"^([a-z_]+):\s*(\S+)", line.strip())
        if m:
            kv[m.group(1)] = m.group(2)
    if kv.get("source_sha") != kernel_source_hash() or kv.get("workload") != workload:
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def algorithmic_bytes(cfg, counts, resident):
    """Bytes the method must move, per SwiGLU expert 3*H*F*b, only activated resident experts count."""
    b = 2 if cfg.dtype == "bf16" else 4
    T, H, E, F, k = cfg.tokens, cfg.hidden, cfg.experts, cfg.ffn, cfg.top_k
    active = [e for e in range(E) if resident[e] and counts[e] > 0]
    n_res = int(sum(counts[e] for e in range(E) if resident[e]))
    n_off = T * k - n_res
    w_expert_p1 = 2 * H * F * b * len(active) + cfg.shared * 2 * H * cfg.shared_ffn * b
    w_expert_all = 3 * H * F * b * len(active) + cfg.shared * 3 * H * cfg.shared_ffn * b
    phase1 = w_expert_p1 + T * H * b                 # W1,W3 of activated experts + the tokens
    layer = w_expert_all + H * E * b + T * H * b + T * H * b + n_off * H * b + T * k * 16
    flops = 6 * H * F * n_res + cfg.shared * 6 * H * cfg.shared_ffn * T + 2 * T * H * E
    return dict(active=len(active), n_res=n_res, n_off=n_off, phase1_bytes=phase1, expert_weight_bytes=w_expert_all,
                layer_bytes=layer, flops=flops, phase1_flops=4 * H * F * n_res + cfg.shared * 4 * H * cfg.shared_ffn * T)


def mfma_peak_tflops(dtype: str) -> float:
    """Dense MFMA peak of the layer's arithmetic type."""
    return MFMA_BF16_PEAK_TFLOPS if dtype == "bf16" else MFMA_F32_PEAK_TFLOPS


def layer_roofline(alg, ms_per_step: float, dtype: str = "bf16"):
    """The whole layer against its roofline: the slower of moving its algorithmic bytes at the HBM
    peak and doing its algorithmic flops at the dense MFMA peak of its type (bf16 or fp32)."""
    t_bytes = alg["layer_bytes"] / (HBM_PEAK_GBPS * 1e9)
    t_flops = alg["flops"] / (mfma_peak_tflops(dtype) * 1e12)
    t_roof = max(t_bytes, t_flops)
    return {"t_roof_us": t_roof * 1e6, "t_bytes_us": t_bytes * 1e6, "t_flops_us": t_flops * 1e6,
            "bound": "hbm" if t_bytes >= t_flops else "mfma", "frac": t_roof / (ms_per_step * 1e-3)}


def cpu_baseline(layer, seconds: float):
    """The CPU oracle (as it stands) on the same layer: whole batches until `seconds` have passed.

    Two more legs, on at most 32 tokens of the batch (routing and repacking still
    cover the whole batch): one thread, and the full layer with the offloaded
    experts too."""
    import numpy as np
    import oracle
    reps = 0
    t0 = time.perf_counter()
    while True:
        oracle.layer_forward_synthetic(layer, offloaded=False)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    toks = reps * layer.cfg.tokens
    n = oracle.threads()
    T = layer.cfg.tokens
    sample = None if T <= 32 else np.arange(32)
    ns = T if sample is None else sample.size
    # the sample on one thread (the oracle's results do not depend on the thread count)
    oracle.set_threads(1)
    t1 = time.perf_counter()
    oracle.layer_forward_synthetic(layer, offloaded=False, sample=sample)
    el1 = time.perf_counter() - t1
    oracle.set_threads(n)
    # the full layer: every pair of the sample, resident or offloaded, after one untimed
    # call that first touches the offloaded experts' weights
    oracle.layer_forward_synthetic(layer, offloaded=True, sample=sample)
    full_reps = 0
    t2 = time.perf_counter()
    while True:
        oracle.layer_forward_synthetic(layer, offloaded=True, sample=sample)
        full_reps += 1
        el2 = time.perf_counter() - t2
        if el2 >= seconds / 10:
            break
    what = "tokens" if sample is None else f"of the first {ns} tokens (FFN; routing and repack over all {T})"
    return {"value": toks / el, "unit": "tokens/s", "cores": n, "kind": "oracle",
            "sample": f"{reps} full batch(es) of {T} tokens of the same layer (resident experts + "
                      f"router + repack, fp64 C with OpenMP), {el:.1f} s",
            "single_thread": {"value": ns / el1, "unit": "tokens/s",
                              "sample": f"1 batch {what} on one thread, {el1:.1f} s"},
            "full_layer": {"value": full_reps * ns / el2, "unit": "tokens/s",
                           "sample": f"{full_reps} batch(es) {what} with the offloaded experts too, {el2:.1f} s"},
            **host_cpu_info()}


def host_cpu_info():
    """CPU model, sockets and cores of this host (from /proc/cpuinfo), and the logical CPUs visible."""
    model, sockets, cores = "unknown", set(), set()
    try:
        with open("/proc/cpuinfo") as f:
            phys = "0"
            for line in f:
                key, _, val = line.partition(":")
                key, val = key.strip(), val.strip()
                if key == "model name" and model == "unknown":
                    model = val
                elif key == "physical id":
                    phys = val
                    sockets.add(val)
                elif key == "core id":
                    cores.add((phys, val))
    except OSError:
        pass
    return {"cpu_model": model, "sockets": len(sockets) or None, "physical_cores": len(cores) or None,
            "logical_cpus_visible": os.cpu_count(), "threads_allowed": len(os.sched_getaffinity(0))}


# rates of this machine (MI355X machine, 16 host threads): host->device copies, the host FFN on
# expert weights and in FLOPs, the device FFN on expert weights -- the cost model's inputs
LINK_GBPS, HOST_GBPS, HOST_GFLOPS, GPU_GBPS = 55.0, 90.0, 500.0, 5900.0


def hybrid_timings(layer, dev, n: int, threads: int, spare: int = 0):
    """Median timings of n hybrid calls: GPU resident/shared experts, host offloaded experts, merge."""
    import numpy as np
    import torch
    import paper_2608_21614_amd as moe
    from paper_2608_21614_amd.device import DeviceLayer
    from paper_2608_21614_amd.hybrid import HybridLayer
    log(f"[bench] hybrid: {n} calls, {threads} host threads, {spare} spare slots")
    rates = None
    if spare > 0:
        c = layer.cfg
        b = 2 if c.dtype == "bf16" else 4
        rates = moe.moe_offload_rates(3 * c.hidden * c.ffn * b, 6 * c.hidden * c.ffn, LINK_GBPS, HOST_GBPS,
                                      HOST_GFLOPS, GPU_GBPS)
        dev = DeviceLayer(layer, n_slots=int(layer.resident.sum()) + spare)
    hy = HybridLayer(dev, layer.w13, layer.w2, threads=threads, rates=rates)
    for _ in range(2):
        hy.forward()
        torch.cuda.synchronize()
    rows = []
    for _ in range(n):
        hy.forward()
        torch.cuda.synchronize()
        rows.append(hy.timings())
    keys = set().union(*[r.keys() for r in rows]) - {"host_t0"}
    med = {k: float(np.median([r.get(k, 0.0) for r in rows])) for k in sorted(keys)}
    med["cost_model"] = None if rates is None else {"link_GBps": LINK_GBPS, "host_GBps": HOST_GBPS,
                                                    "host_GFLOPs": HOST_GFLOPS, "gpu_GBps": GPU_GBPS,
                                                    "spare_slots": spare}
    c = layer.cfg
    b = 2 if c.dtype == "bf16" else 4
    cnt, seg, nres = hy.h_counts.numpy(), hy.h_seg.numpy(), int(hy.h_nres[0])
    n_off_experts = int(((cnt > 0) & (seg >= nres)).sum())      # experts the host ran in the last call
    host_bytes = n_off_experts * 3 * c.hidden * c.ffn * b
    med["host_experts"] = n_off_experts
    med["host_weight_bytes"] = host_bytes
    med["host_ffn_GBps"] = host_bytes / (med["host_ffn_ms"] * 1e-3) / 1e9 if med["host_ffn_ms"] > 0 else None
    med["threads"] = threads
    return med


def bookkeeping_timings(dev, n: int):
    """Median wall time per synchronised call: fused repacked forward vs the bookkeeping baseline."""
    import numpy as np
    import torch
    from paper_2608_21614_amd.bookkeeping import BookkeepingLayer
    log(f"[bench] bookkeeping A/B: {n} calls each")
    bk = BookkeepingLayer(dev)
    o = dev.alloc_outputs()
    args = dev.args(o)
    import paper_2608_21614_amd as moe

    def fused():
        moe.moe_layer_forward(args, dev.ws)

    def timed(fn):
        ts = []
        for i in range(n + 3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            if i >= 3:
                ts.append((time.perf_counter() - t0) * 1e3)
        return float(np.median(ts))

    f_ms = timed(fused)
    b_ms = timed(bk.forward)
    return {"fused_ms": f_ms, "bookkeeping_ms": b_ms, "speedup": b_ms / f_ms,
            "resident_experts": len(bk.resident), "host_syncs_per_call": bk.last["host_syncs"],
            "timing": "wall clock per call, device synchronised before and after each call"}


def trace_timings(seed: int, lags, detect: bool = False, persistence: float = 0.0):
    """The stage-structured decode trace with real slot copies (Section IV-C), per prefetch lag.

    Routers, stage biases and per-call activations are the trace's own (so the
    residency trajectory and CHR are the ones the parity tests check).  With
    `detect`, the boundaries come from the cue machine on the batch's generated
    tokens (Section IV-B.1) instead of the trace's true stage ends.  Every
    (layer, expert) gets its own pinned host buffer filled with one seeded
    expert's weights -- the values do not change routing, copies or kernel time.
    """
    import numpy as np
    import torch
    from paper_2608_21614_amd.device import to_device
    from paper_2608_21614_amd.residency import StageResidencyRunner
    from dataclasses import replace
    from workloads import TRACE, StageTrace
    c = replace(TRACE, stage_persistence=persistence)
    trace = StageTrace(c, seed=seed)
    L, E = c.layers, c.experts
    layers = [trace.layer(l, cache_weights=False) for l in range(L)]
    log(f"[bench] trace: {c.steps} steps x {L} layers, {trace.n_stages} stages; generating inputs")
    xs = []
    for l in range(L):
        xs.append(to_device(np.stack([trace.x(s, l) for s in range(c.steps)])))   # [steps, T, H] on the device
    base13, base2 = layers[0].w13(0), layers[0].w2(0)
    out = {"steps": c.steps, "layers": L, "stages": int(trace.n_stages), "batch": c.batch, "slots": c.n_slots,
           "stage_persistence": persistence,
           "weights": "one seeded expert's weights in every (layer, expert) host buffer", "runs": []}
    detector = None
    if detect:
        ts = trace.token_stream()
        detector = {"cues": ts["cues"], "stream": ts["stream"]}
        out["boundaries"] = "detected from cues in the generated tokens"
        out["planted_boundaries"] = int(len(ts["planted"]))
    runner = None
    for lag in lags:
        log(f"[bench] trace run, prefetch lag {lag}")
        if runner is None:
            runner = StageResidencyRunner(trace, [lay.w_router for lay in layers], lambda l, e: (base13, base2),
                                          lambda s, l: xs[l][s], lag=lag)
            runner.prepare_host_weights()
        else:   # same host buffers and slot pools, fresh trajectory
            runner.reset(lag)
        r = runner.run(detector=detector)
        calls = r["calls"]
        if "tc_seq" not in out:   # routing, hence the stage activation matrices, does not depend on the lag
            from paper_2608_21614_amd.stage_trace import clairvoyant_chr, temporal_coherence
            out["tc_seq"] = temporal_coherence(r["counts"], trace.stage_len)
            out["chr_clairvoyant"] = clairvoyant_chr(r["counts"], trace.stage_len, c.n_slots)
            if detect:
                edges = np.concatenate([[0], r["boundary_steps"] + 1, [c.steps]])
                out["tc_seq_detected_stages"] = temporal_coherence(r["counts"], np.diff(edges))
        out["runs"].append({"lag": lag, "trace_ms": r["trace_ms"], "us_per_layer_call": r["trace_ms"] * 1e3 / calls,
                            "chr_online": r["chr_online"], "copied_experts": r["copied_experts"],
                            "copy_ms_total": r["copy_ms_total"], "copy_GBps": r["copy_GBps"],
                            "stall_ms_total": r["stall_ms_total"], "boundaries": int(len(r["boundary_steps"])),
                            "eta_chr": r["chr_online"] / out["chr_clairvoyant"]})
        log(f"[bench]   {out['runs'][-1]}")
    return out


def _time_layer_calls(dev, steps: int, warmup: int, rotate_bytes: int = 1 << 30, max_copies: int = 32,
                      pack_offloaded: bool = True):
    """Mean wall time per fused call of `dev` over `steps` calls (after `warmup`), rotating
    enough copies of its expert weights (routed and shared) that each call reads at least
    `rotate_bytes` of other weights before its own come round again; then the mean FFN
    phase-1 duration from the library's stage events over min(steps, 50) more calls.
    Returns (us per call, phase-1 us, counts, weight copies)."""
    import numpy as np
    import torch
    import paper_2608_21614_amd as moe
    from paper_2608_21614_amd.device import to_host

    per_copy = sum(t.numel() * t.element_size() for t in (dev.w13, dev.w2, dev.ws13, dev.ws2) if t is not None)
    n_copies = int(min(max_copies, max(4, -(-rotate_bytes // max(per_copy, 1)))))
    base = (dev.w13, dev.w2, dev.ws13, dev.ws2)
    copies = [base] + [tuple(None if t is None else t.clone() for t in base) for _ in range(n_copies - 1)]
    o = dev.alloc_outputs()

    def make_args(i, events=None):
        dev.w13, dev.w2, dev.ws13, dev.ws2 = copies[i % n_copies]
        a = dev.args(o, pack_offloaded=pack_offloaded)
        if events is not None:
            a.stage_events = ctypes.cast(events, ctypes.POINTER(ctypes.c_void_p))
        return a

    plain = [make_args(i) for i in range(n_copies)]
    hip = moe.hip_runtime()
    hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    nE = moe.MOE_STAGE_EVENTS
    P1_BEFORE, P1_AFTER = 3, 4
    n_ev = min(steps, 50)
    evs, created = [], []
    for _ in range(n_ev):
        arr = (ctypes.c_void_p * nE)()
        for j in (P1_BEFORE, P1_AFTER):
            ev = ctypes.c_void_p()
            assert hip.hipEventCreateWithFlags(ctypes.byref(ev), 0) == 0
            created.append(ev.value)
            arr[j] = ev.value
        evs.append(arr)
    with_ev = [make_args(i, evs[i]) for i in range(n_ev)]
    dev.w13, dev.w2, dev.ws13, dev.ws2 = base
    stream = torch.cuda.current_stream()
    for i in range(warmup):
        moe.moe_layer_forward(plain[i % n_copies], dev.ws, stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        moe.moe_layer_forward(plain[i % n_copies], dev.ws, stream)
    torch.cuda.synchronize()
    us = (time.perf_counter() - t0) * 1e6 / max(steps, 1)
    for a in with_ev:
        moe.moe_layer_forward(a, dev.ws, stream)
    torch.cuda.synchronize()
    f = ctypes.c_float()
    p1 = []
    for arr in evs:
        assert hip.hipEventElapsedTime(ctypes.byref(f), arr[P1_BEFORE], arr[P1_AFTER]) == 0
        p1.append(f.value * 1e3)
    for e in created:
        hip.hipEventDestroy(e)
    counts = to_host(o["counts"])
    del copies, plain, with_ev, o
    return us, float(np.mean(p1)) if p1 else 0.0, counts, n_copies


def ep_shard_timings(layer, n: int, steps: int, warmup: int):
    """One GPU's share of the layer under n-way expert parallelism, each shard timed on this
    GPU as its own fused call, beside the whole layer with every expert resident on one GPU.

    Routing is replicated (every shard routes the whole batch); shard g holds a contiguous
    block of routed expert ids and a 64-column slice of each shared expert, and packs no
    offloaded rows (the other experts are other GPUs' work).  What one GPU cannot show is
    left out: the cross-GPU sum of the shards' [T, H] partial outputs is neither built nor
    timed, so the slowest shard is a lower bound on an n-GPU layer call.
    """
    import numpy as np
    import torch
    from paper_2608_21614_amd.device import DeviceLayer
    from workloads import ExpertShard

    c = layer.cfg
    log(f"[bench] {c.name}: {n}-way expert-parallel shards")
    whole = ExpertShard(layer, 1, 0)
    dev = DeviceLayer(whole)
    one_us, one_p1, _, one_copies = _time_layer_calls(dev, steps, warmup, pack_offloaded=False)
    del dev
    torch.cuda.empty_cache()
    shards = []
    for g in range(n):
        sh = ExpertShard(layer, n, g)
        dev = DeviceLayer(sh)
        us, p1, cnt, nc = _time_layer_calls(dev, steps, warmup, pack_offloaded=False)
        del dev
        torch.cuda.empty_cache()
        alg = algorithmic_bytes(sh.cfg, cnt, sh.resident)
        rec = {"shard": g, "experts": [int(sh.expert_ids[0]), int(sh.expert_ids[-1]) + 1] if sh.n_slots else [],
               "shared_cols": list(sh.shared_cols), "pairs": alg["n_res"], "active_experts": alg["active"],
               "us_per_call": us, "ffn_phase1_us": p1, "weight_copies": nc}
        if c.tokens > 64:
            rec["ffn_phase1_TFLOPs"] = alg["phase1_flops"] / (p1 * 1e-6) / 1e12
        else:
            rec["ffn_phase1_GBps"] = alg["phase1_bytes"] / (p1 * 1e-6) / 1e9
        shards.append(rec)
    t = np.array([r["us_per_call"] for r in shards])
    return {"n": n, "split": "routed experts in contiguous id blocks; shared experts by 64-column FFN slices; "
                             "routing replicated; no offloaded-row pack",
            "one_gpu_all_resident_us": one_us, "one_gpu_all_resident_ffn_phase1_us": one_p1,
            "one_gpu_weight_copies": one_copies,
            "max_shard_us": float(t.max()), "mean_shard_us": float(t.mean()), "imbalance": float(t.max() / t.mean()),
            "speedup_of_slowest_shard": one_us / float(t.max()),
            "not_built": "the cross-GPU reduction of the shards' partial outputs", "shards": shards}


# the configs measured besides the primary one in a default run (each with its own
# roofline and a bounded CPU-oracle sample): the tiny fp32 layer, the shared+routed
# decode batch, the prefill chunk, one layer call of the stage-structured trace, and
# the Qwen3-MoE-like decode batch (and c4's shape in fp32)
OTHER_WORKLOADS = ["c1_tiny_f32", "c3_shared_decode", "c4_prefill", "c5_stage_trace", "c6_qwen3_decode",
                   "c4_prefill_f32"]


def measure_workload(name, cfg, args, steps: int, warmup: int, cpu_seconds: float, primary: bool,
                     read_probe_gbps=None):
    """Times `steps` fused layer forwards of one workload (after `warmup` untimed ones) and
    returns its measurement: step time, tokens/s, the dominant kernel's roofline, the whole
    layer's roofline, the per-stage breakdown and (unless disabled) the CPU oracle's rate."""
    import numpy as np
    import torch

    import paper_2608_21614_amd as moe
    from paper_2608_21614_amd.device import DeviceLayer, to_host
    from workloads import SyntheticLayer

    log(f"[bench] generating {name} seed {args.seed}")
    layer = SyntheticLayer(cfg, args.seed)
    dev = DeviceLayer(layer)
    copies = [(dev.w13, dev.w2)] + [(dev.w13.clone(), dev.w2.clone()) for _ in range(args.copies - 1)]
    o = dev.alloc_outputs()
    hip = moe.hip_runtime()
    hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    created = []

    def new_event():
        ev = ctypes.c_void_p()
        assert hip.hipEventCreateWithFlags(ctypes.byref(ev), 0) == 0
        created.append(ev.value)
        return ev

    nE = moe.MOE_STAGE_EVENTS
    P1_BEFORE, P1_AFTER = 3, 4  # stage events around FFN phase 1
    # every EVENT_EVERY-th timed step records the two events around the dominant
    # kernel (each event record costs GPU time, about 2.5 us); a separate untimed
    # pass records every stage boundary
    timed_ev = [i for i in range(steps) if i % EVENT_EVERY == 0]
    ev = {i: (ctypes.c_void_p * nE)(*[new_event().value if j in (P1_BEFORE, P1_AFTER) else None for j in range(nE)])
          for i in timed_ev}
    n_diag = min(steps, 50)
    ev_all = [(ctypes.c_void_p * nE)(*[new_event().value for _ in range(nE)]) for _ in range(n_diag)]

    def make_args(i, events=None):
        w13, w2 = copies[i % len(copies)]
        dev.w13, dev.w2 = w13, w2
        a = dev.args(o)
        if events is not None:
            a.stage_events = ctypes.cast(events, ctypes.POINTER(ctypes.c_void_p))
        return a

    plain = [make_args(i) for i in range(len(copies))]
    timed = [make_args(i, ev.get(i)) for i in range(steps)]
    diag = [make_args(i, ev_all[i]) for i in range(n_diag)]
    stream = torch.cuda.current_stream()

    if primary and args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {args.calib_copy_mib} MiB done")
        del src, dst

    for i in range(warmup):
        moe.moe_layer_forward(plain[i % len(plain)], dev.ws, stream)
    torch.cuda.synchronize()
    log(f"[bench] {name}: warmup {warmup} done; timing {steps} steps")
    t0 = time.perf_counter()
    for i in range(steps):
        moe.moe_layer_forward(timed[i], dev.ws, stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    f = ctypes.c_float()
    p1_ms = np.zeros(len(timed_ev))
    for n, i in enumerate(timed_ev):
        assert hip.hipEventElapsedTime(ctypes.byref(f), ev[i][P1_BEFORE], ev[i][P1_AFTER]) == 0
        p1_ms[n] = f.value

    # untimed diagnostics: every stage boundary instrumented, and steps with no events at all
    for i in range(n_diag):
        moe.moe_layer_forward(diag[i], dev.ws, stream)
    torch.cuda.synchronize()
    stage_ms = np.zeros((n_diag, nE - 1))
    for i in range(n_diag):
        for j in range(nE - 1):
            assert hip.hipEventElapsedTime(ctypes.byref(f), ev_all[i][j], ev_all[i][j + 1]) == 0
            stage_ms[i, j] = f.value
    stage_us = {n: float(stage_ms[:, j].mean() * 1e3) for j, n in enumerate(STAGES)}
    step_us = stage_ms.sum(axis=1) * 1e3       # per instrumented step: first to last stage event
    step_pct = {"p10": float(np.percentile(step_us, 10)), "median": float(np.median(step_us)),
                "p90": float(np.percentile(step_us, 90)), "steps": int(n_diag)}
    t1 = time.perf_counter()
    for i in range(steps):
        moe.moe_layer_forward(plain[i % len(plain)], dev.ws, stream)
    torch.cuda.synchronize()
    ms_no_events = (time.perf_counter() - t1) * 1e3 / steps

    ms_graph = None
    if primary:
        # the same calls replayed from a HIP graph: one capture of one call per weight copy
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            for a in plain:
                moe.moe_layer_forward(a, dev.ws)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for a in plain:
                moe.moe_layer_forward(a, dev.ws)
        reps = max(1, steps // len(plain))
        graph.replay()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        for _ in range(reps):
            graph.replay()
        torch.cuda.synchronize()
        ms_graph = (time.perf_counter() - t2) * 1e3 / (reps * len(plain))
        del graph

    if read_probe_gbps is None:
        # streaming-read reference of this GPU: one pass of 16-byte loads over 4 GiB
        probe_src = torch.empty(1 << 30, dtype=torch.float32, device="cuda")
        probe_sink = torch.zeros(1, dtype=torch.int32, device="cuda")
        pe0, pe1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(2):
            moe.moe_read_probe(probe_src, probe_sink, stream=stream)
        pe0.record(stream)
        for _ in range(10):
            moe.moe_read_probe(probe_src, probe_sink, stream=stream)
        pe1.record(stream)
        torch.cuda.synchronize()
        read_probe_gbps = 10 * probe_src.numel() * 4 / (pe0.elapsed_time(pe1) * 1e-3) / 1e9
        del probe_src, probe_sink

    counts = to_host(o["counts"])
    resident = (layer.expert_slot >= 0) & (layer.expert_slot < dev.slots)
    alg = algorithmic_bytes(cfg, counts, resident)
    ms_per_step = wall * 1e3 / steps
    tokens_per_s = cfg.tokens / (ms_per_step * 1e-3)
    p1_us = float(p1_ms.mean() * 1e3)
    p1_pct = {"p10": float(np.percentile(p1_ms, 10) * 1e3), "median": float(np.median(p1_ms) * 1e3),
              "p90": float(np.percentile(p1_ms, 90) * 1e3)}
    p1_s = p1_us * 1e-6
    traffic = read_traffic(name)
    if cfg.tokens > 64:
        # prefill-size batches run MFMA kernels at the ridge (bf16: the tiled kernel; fp32: the
        # stream kernel over 64-row chunks): FLOP rate against the dense matrix-core peak of the
        # layer's type, and the HBM fraction beside it
        achieved = alg["phase1_flops"] / p1_s / 1e12
        peak = mfma_peak_tflops(cfg.dtype)
        kname = ("k_ffn_tiled (phase 1: gate/up projections + SwiGLU)" if cfg.dtype == "bf16" else
                 "k_ffn_stream fp32, 64-row chunks (phase 1: gate/up projections + SwiGLU)")
        roofline = {"kernel": kname, "bound": "mfma",
                    "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                    "frac": achieved / peak, "traffic": traffic,
                    "algorithmic_flops_per_launch": alg["phase1_flops"],
                    "algorithmic_bytes_per_launch": alg["phase1_bytes"],
                    "hbm_frac_algorithmic": alg["phase1_bytes"] / p1_s / 1e9 / HBM_PEAK_GBPS, "mean_launch_us": p1_us,
                    "launch_us": p1_pct, "launches_timed": len(timed_ev)}
    else:
        achieved = alg["phase1_bytes"] / p1_s / 1e9
        roofline = {"kernel": "k_ffn_stream (phase 1: gate/up projections + SwiGLU)", "bound": "hbm",
                    "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBPS,
                    "read_probe_GBps": read_probe_gbps, "frac_of_read_probe": achieved / read_probe_gbps,
                    "traffic": traffic, "algorithmic_bytes_per_launch": alg["phase1_bytes"], "mean_launch_us": p1_us,
                    "launch_us": p1_pct, "launches_timed": len(timed_ev)}
    m = {
        "workload": name,
        "description": cfg.description,
        "dtype": "bf16" if cfg.dtype == "bf16" else "f32",
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "tokens_per_s": tokens_per_s,
        "shape": {"tokens": cfg.tokens, "hidden": cfg.hidden, "experts": cfg.experts, "ffn": cfg.ffn,
                  "top_k": cfg.top_k, "shared": cfg.shared, "shared_ffn": cfg.shared_ffn,
                  "resident_slots": dev.slots, "active_resident_experts": alg["active"],
                  "resident_pairs": alg["n_res"], "offloaded_pairs": alg["n_off"], "seed": args.seed,
                  "weight_copies": len(copies)},
        "hbm_gbps_expert_weights": alg["expert_weight_bytes"] / (ms_per_step * 1e-3) / 1e9,
        "hbm_gbps_layer_algorithmic": alg["layer_bytes"] / (ms_per_step * 1e-3) / 1e9,
        "mfma_tflops_layer_algorithmic": alg["flops"] / (ms_per_step * 1e-3) / 1e12,
        "stages_us_instrumented": stage_us,
        "step_us_instrumented": step_pct,
        "ms_per_step_without_events": ms_no_events,
        # whole layer against its roofline: the slower of moving its algorithmic bytes at
        # the HBM peak and doing its algorithmic flops at the dense bf16 MFMA peak
        "layer_roofline": layer_roofline(alg, ms_per_step, cfg.dtype),
        "roofline": roofline,
        "hbm_read_probe_GBps": read_probe_gbps,
    }
    if ms_graph is not None:
        # the same calls replayed from a HIP graph (one graph launch per call instead of 5-6 kernel launches)
        m["ms_per_step_graph"] = ms_graph
    if primary and args.bookkeeping > 0:
        m["bookkeeping"] = bookkeeping_timings(dev, args.bookkeeping)
    if primary and args.hybrid > 0:
        m["hybrid"] = hybrid_timings(layer, dev, args.hybrid, args.host_threads, args.hybrid_spare)
    for e in created:
        hip.hipEventDestroy(e)
    del copies, dev, o, plain, timed, diag
    torch.cuda.empty_cache()
    if args.ep > 1:
        m["ep_shards"] = ep_shard_timings(layer, args.ep, min(steps, 100), warmup)
    if cpu_seconds > 0:
        log(f"[bench] {name}: timing the CPU oracle ({cpu_seconds:.0f} s sample)")
        m["cpu_baseline"] = cpu_baseline(layer, cpu_seconds)
    return m


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="c2_mixtral_decode",
                    help="the primary workload, whose throughput is `value`")
    ap.add_argument("--only", action="store_true",
                    help="measure the primary workload only (default: the other configs follow, each as an "
                         "entry of `workloads`)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copies", type=int, default=4, help="rotated expert-weight copies")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--other-cpu-seconds", type=float, default=3.0,
                    help="CPU-oracle sample per other config (0: none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--hybrid", type=int, default=0, metavar="N",
                    help="also time N hybrid layer calls (offloaded experts on the host, Section IV-D.2); "
                         "reported as an extra object, `value` stays the GPU path")
    ap.add_argument("--host-threads", type=int, default=16)
    ap.add_argument("--hybrid-spare", type=int, default=0, metavar="S",
                    help="with --hybrid: S spare device slots and the per-expert cost model (copy vs host)")
    ap.add_argument("--bookkeeping", type=int, default=0, metavar="N",
                    help="also time N calls of the bookkeeping baseline (per-expert mask/gather/FFN/scatter) "
                         "against N fused calls, each synchronised; extra object")
    ap.add_argument("--trace", type=str, default="", metavar="LAGS",
                    help="with --workload c5_stage_trace: also run the whole stage-structured trace with real "
                         "slot copies, once per comma-separated prefetch lag (e.g. 0,8); extra object")
    ap.add_argument("--trace-persistence", type=float, default=0.0, metavar="RHO",
                    help="with --trace: each stage's expert popularity is RHO x the previous stage's + (1 - RHO) x "
                         "a fresh Dirichlet draw (0, the default: independent stages)")
    ap.add_argument("--detect", action="store_true",
                    help="with --trace: stage boundaries from the cue machine on the generated tokens "
                         "(Section IV-B.1) instead of the trace's true stage ends")
    ap.add_argument("--ep", type=int, default=8, metavar="N",
                    help="also time each GPU's share of every measured workload under N-way expert parallelism "
                         "(each shard as its own call on this GPU) beside the all-resident one-GPU call; "
                         "extra object, 0 or 1: off")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (counter calibration)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build measures one GPU only: the MoE-layer hot path runs on one "
                                   "MI355X; multi-GPU sharding is a design note, not built"}), flush=True)
        return 2

    import torch

    from workloads import CONFIGS, TRACE

    # the stage-structured trace's layer shape is timed as one layer call (no stage bias)
    cfgs = dict(CONFIGS)
    cfgs[TRACE.name] = TRACE.layer_config()
    if args.workload not in cfgs:
        print(json.dumps({"error": f"unknown workload {args.workload}; one of {sorted(cfgs)}"}), flush=True)
        return 2
    cfg = cfgs[args.workload]
    torch.cuda.set_device(0)
    cpu_s = 0.0 if args.no_cpu_baseline else args.cpu_seconds
    m = measure_workload(args.workload, cfg, args, args.steps, args.warmup, cpu_s, primary=True)
    result = {
        "metric": METRIC,
        "value": m["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": m["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": m["dtype"],
        "data": f"synthetic (seeded: x ~ N(0,1), weights ~ N(0,0.02^2), {cfg.dtype})",
        "config": {"workload": args.workload, "description": cfg.description, **m["shape"], "parallelism": "1 GPU"},
    }
    for key in ("hbm_gbps_expert_weights", "hbm_gbps_layer_algorithmic", "stages_us_instrumented",
                "step_us_instrumented", "ms_per_step_without_events", "ms_per_step_graph", "hbm_read_probe_GBps",
                "mfma_tflops_layer_algorithmic", "layer_roofline", "roofline", "bookkeeping", "hybrid", "ep_shards"):
        if key in m:
            result[key] = m[key]
    if not args.only:
        # every other config, one after another in the same process: same step count,
        # same weight rotation, a shorter CPU-oracle sample each
        other_cpu = 0.0 if args.no_cpu_baseline else args.other_cpu_seconds
        result["workloads"] = {}
        for name in OTHER_WORKLOADS:
            if name == args.workload:
                continue
            result["workloads"][name] = measure_workload(name, cfgs[name], args, args.steps, args.warmup, other_cpu,
                                                         primary=False, read_probe_gbps=m["hbm_read_probe_GBps"])
    if args.trace:
        torch.cuda.empty_cache()
        result["trace"] = trace_timings(args.seed, [int(v) for v in args.trace.split(",")], args.detect,
                                        args.trace_persistence)
    if "cpu_baseline" in m:
        result["cpu_baseline"] = m["cpu_baseline"]
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
