"""Hybrid CPU-GPU layer (SAEM Section IV-D.2): full layer output vs the oracle.

Resident and shared experts run on the GPU, offloaded experts on the host
(moe_host_ffn over the packed rows the GPU copied out), and moe_combine merges
both.  The result must be the oracle's complete layer (out_res + out_off) under
the routing the GPU chose (near ties resolved as in the other parity tests).
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from gpu_support import DELTA, TOL, expected_routing, host_f64, rel_l2
from workloads import CONFIGS, SyntheticLayer

pytestmark = pytest.mark.gpu


def say(*a):
    print("[hybrid]", *a, flush=True)


def run_hybrid(lay, sample=None, threads=16, rates=None, spare_slots=0):
    from paper_2608_21614_amd.device import DeviceLayer, to_host
    from paper_2608_21614_amd.hybrid import HybridLayer
    c = lay.cfg
    dev = DeviceLayer(lay, n_slots=int(lay.resident.sum()) + spare_slots)
    hy = HybridLayer(dev, lay.w13, lay.w2, threads=threads, rates=rates)
    out = hy.forward()
    torch.cuda.synchronize()
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    lg = to_host(hy.o["logits"]).astype(np.float64)
    assert np.abs(lg - lg_ref).max() < DELTA / 2
    idx = to_host(hy.o["topk_idx"])
    exp_idx, _ = expected_routing(lg_ref, idx, c.top_k)
    np.testing.assert_array_equal(idx, exp_idx)
    ref = oracle.layer_forward_synthetic(lay, idx=exp_idx, sample=sample, offloaded=True)
    n_res = int(to_host(hy.o["n_res"])[0])
    # resident pairs under the map the call ran with (the base map, plus any experts copied in)
    call_map = to_host(hy.d_map)
    resident = (call_map >= 0) & (call_map < dev.slots)
    assert n_res == int(np.bincount(exp_idx.ravel(), minlength=c.experts)[resident].sum())
    if not hy.last.get("copied_experts"):
        assert n_res == ref["n_res"]
    full = ref["out_res"] + ref["out_off"]
    got = host_f64(out)[ref["sample"]]
    err = rel_l2(got, full)
    say(f"{c.name}: n_off {c.tokens * c.top_k - n_res}, full-output rel-L2 {err:.3e}, timings {hy.timings()}")
    return err, n_res, hy


SMALL = replace(CONFIGS["c2_mixtral_decode"], name="small_bf16", tokens=24, hidden=256, experts=8, ffn=192,
                top_k=2, n_resident=4)


@pytest.mark.parametrize("seed", [0, 1])
def test_hybrid_small_full_output(seed):
    say("small bf16 seed", seed)
    err, n_res, _ = run_hybrid(SyntheticLayer(SMALL, seed))
    assert n_res < SMALL.tokens * SMALL.top_k
    assert err <= TOL["bf16"]


def test_hybrid_small_f32_full_output():
    cfg = replace(SMALL, name="small_f32", dtype="f32", tokens=16, hidden=128, ffn=128)
    say("small f32")
    err, n_res, _ = run_hybrid(SyntheticLayer(cfg, 2))
    assert n_res < cfg.tokens * cfg.top_k
    assert err <= TOL["f32"]


def test_hybrid_repeated_calls_are_identical():
    """The same inputs twice: bitwise-equal outputs (fixed-order GPU sums, per-element host sums)."""
    from paper_2608_21614_amd.device import DeviceLayer
    from paper_2608_21614_amd.hybrid import HybridLayer
    lay = SyntheticLayer(SMALL, 3)
    hy = HybridLayer(DeviceLayer(lay), lay.w13, lay.w2, threads=4)
    a = hy.forward().clone()
    b = hy.forward().clone()
    torch.cuda.synchronize()
    assert torch.equal(a, b)


@pytest.mark.parametrize("name,seed", [("c2_mixtral_decode", 0), ("c3_shared_decode", 1)])
def test_hybrid_full_size(name, seed):
    say(name, "seed", seed, "(every token)")
    lay = SyntheticLayer(CONFIGS[name], seed)
    err, n_res, _ = run_hybrid(lay)
    assert n_res < lay.cfg.tokens * lay.cfg.top_k
    assert err <= TOL["bf16"]


def test_hybrid_cost_model_copies_busy_experts():
    """With a slow host (compute-bound at 1 GFLOP/s) the cost model copies the busiest offloaded
    experts into the two spare slots; the full layer output is unchanged."""
    import paper_2608_21614_amd as moe
    cfg = replace(SMALL, name="small_copy", tokens=64, top_k=4, n_resident=3)
    H, F = cfg.hidden, cfg.ffn
    rates = moe.moe_offload_rates(3 * H * F * 2, 6 * H * F, 50.0, 50.0, 1.0, 5000.0)
    say("cost model: copies to spare slots")
    err, n_res, hy = run_hybrid(SyntheticLayer(cfg, 0), rates=rates, spare_slots=2)
    assert hy.last["copied_experts"] == 2
    assert err <= TOL["bf16"]
    # the two copied experts sit in the spare slots 3 and 4 of this call's map
    from paper_2608_21614_amd.device import to_host
    assert sorted(int(v) for v in to_host(hy.d_map) if v >= 3) == [3, 4]
