"""GPU parity of the stage-structured decode trace (2048 steps x 8 layers x 16
tokens, Mixtral-style routers, Dirichlet stage biases, 2 of 8 experts resident
per layer): routing, repacking, the per-stage activation log, the residency
plan at every stage boundary and the cache-hit ratio against the oracle; the
full layer forward on sampled calls."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle
from gpu_support import TOL, expected_routing, host_f64, rel_l2
from workloads import TRACE, StageTrace, SyntheticLayer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_21614_amd as m
    return m


def say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(scope="module")
def trace_run(moe):
    """The whole trace on the GPU (routing, logs, plans) and the oracle's counts and replay."""
    from paper_2608_21614_amd.stage_trace import run_routing_trace
    cfg = TRACE
    trace = StageTrace(cfg, seed=0)
    L, T, E, k, H = cfg.layers, cfg.batch, cfg.experts, cfg.top_k, cfg.hidden
    say(f"trace: {cfg.steps} steps x {L} layers x {T} tokens, {trace.n_stages} stages")
    layers = [trace.layer(l, cache_weights=False) for l in range(L)]
    routers = [lay.w_router for lay in layers]
    xs = [np.stack([trace.x(s, l) for s in range(cfg.steps)]) for l in range(L)]   # [steps, T, H] per layer
    say("inputs generated")
    gpu = run_routing_trace(trace, routers, x_of=lambda s, l: xs[l][s], log_every=512)
    say(f"GPU trace done, online CHR {gpu['chr_online']:.4f}")

    stage_of = trace.stage_of_step()
    counts = np.empty((cfg.steps, L, E), dtype=np.int64)
    for l in range(L):
        lg = oracle.router_logits(xs[l].reshape(-1, H), routers[l], None)
        lg = lg + np.repeat(trace.stage_bias[stage_of, l].astype(np.float64), T, axis=0)
        idx_gpu = gpu["topk_idx"][:, l].reshape(-1, k)
        exp_idx, alts = expected_routing(lg, idx_gpu, k)
        np.testing.assert_array_equal(idx_gpu, exp_idx)
        for s in range(cfg.steps):
            counts[s, l] = oracle.repack(exp_idx[s * T:(s + 1) * T], np.ones(E, bool))["counts"]
        say(f"layer {l}: routing exact ({len(alts)} near-tied tokens)")

    init = np.full((L, E), -1, np.int32)
    for l in range(L):
        ids = np.flatnonzero(trace.initial_resident[l])
        init[l, ids] = np.arange(len(ids))
    ref = oracle.stage_replay(counts, trace.stage_len, init, cfg.n_slots)
    return {"trace": trace, "xs": xs, "gpu": gpu, "counts": counts, "ref": ref, "stage_of": stage_of}


def test_stage_trace_residency_and_chr(trace_run):
    gpu, counts, ref = trace_run["gpu"], trace_run["counts"], trace_run["ref"]
    np.testing.assert_array_equal(gpu["counts"], counts)
    np.testing.assert_array_equal(gpu["slot_history"], ref["slot_history"])
    res_pairs = (counts * ref["resident"]).sum(axis=2)
    np.testing.assert_array_equal(gpu["n_res"], res_pairs)
    assert gpu["chr_online"] == ref["chr_online"]
    say(f"CHR online {ref['chr_online']:.4f}, clairvoyant {ref['chr_clairvoyant']:.4f}, eta {ref['eta_chr']:.4f}")


def test_stage_trace_forward_first_and_last_step_of_every_stage(trace_run):
    """The full layer forward (resident partial) at the first and the last step of
    every stage, for the first and the last layer, with the residency in effect at
    that step; every token's output is checked."""
    from paper_2608_21614_amd.device import DeviceLayer, to_host
    cfg = TRACE
    trace, xs, gpu, ref, stage_of = (trace_run[n] for n in ("trace", "xs", "gpu", "ref", "stage_of"))
    ends = [int(v) for v in trace.stage_ends()]
    firsts = [0] + [e + 1 for e in ends[:-1]]
    for l in (0, cfg.layers - 1):
        lay = SyntheticLayer(cfg.layer_config(), 0, layer=l)      # expert weights cached across the calls
        for s in range(trace.n_stages):
            for step in sorted({firsts[s], ends[s]}):
                assert int(stage_of[step]) == s
                lay.x = xs[l][step]
                lay.bias = trace.stage_bias[s, l].copy()
                slot = ref["slot_history"][s, l]
                lay.set_residency(slot >= 0, expert_slot=slot)
                dev = DeviceLayer(lay)
                o = dev.alloc_outputs()
                dev.forward(o)
                torch.cuda.synchronize()
                idx = to_host(o["topk_idx"])
                np.testing.assert_array_equal(idx, gpu["topk_idx"][step, l])
                out = oracle.layer_forward_synthetic(lay, idx=idx, offloaded=False)
                np.testing.assert_array_equal(to_host(o["counts"]), out["counts"])
                assert int(to_host(o["n_res"])[0]) == int(gpu["n_res"][step, l])
                err = rel_l2(host_f64(o["out"]), out["out_res"])
                say(f"  layer {l} stage {s} step {step}: resident {np.flatnonzero(slot >= 0).tolist()}, "
                    f"rel-L2 {err:.3e}")
                assert err <= TOL["bf16"]
                del dev, o
        del lay
        torch.cuda.empty_cache()
