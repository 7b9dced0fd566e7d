"""One GPU's share of a layer under expert parallelism, run through the C ABI.

Each shard (``workloads.ExpertShard``: a contiguous block of routed experts and
a 64-column slice of every shared expert) runs as its own fused layer call with
fp32 output and no offloaded-row pack.  The shards' partial outputs, summed on
the host in shard order, must match the oracle's whole-layer output (every
routed expert plus the shared experts) at the layer's bar; every shard must
route the batch identically.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_support import TOL, expected_routing, host_f64, rel_l2
from workloads import CONFIGS, ExpertShard, SyntheticLayer, make_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_21614_amd as m
    return m


def say(*a):
    print("[case]", *a, flush=True)
    sys.stdout.flush()


def run_shards(moe, lay, n, sample):
    from paper_2608_21614_amd.device import DeviceLayer, to_host
    total, idx0, counts0 = None, None, None
    for g in range(n):
        sh = ExpertShard(lay, n, g)
        dev = DeviceLayer(sh)
        o = dev.alloc_outputs(out_dtype=moe.MOE_F32)
        moe.moe_layer_forward(dev.args(o, pack_offloaded=False), dev.ws)
        torch.cuda.synchronize()
        idx, counts = to_host(o["topk_idx"]), to_host(o["counts"])
        if g == 0:
            idx0, counts0 = idx, counts
        np.testing.assert_array_equal(idx, idx0)
        np.testing.assert_array_equal(counts, counts0)
        assert int(to_host(o["n_res"])[0]) == int(counts[sh.expert_ids].sum())
        part = host_f64(o["out"])[sample]
        total = part if total is None else total + part
        del dev, o
    return total, idx0


@pytest.mark.parametrize("name,n,n_sample", [("c1_tiny_f32", 8, None), ("c2_mixtral_decode", 8, None),
                                             ("c3_shared_decode", 8, None), ("c6_qwen3_decode", 8, None),
                                             ("c4_prefill", 8, 256), ("c4_prefill_f32", 8, 128),
                                             ("c3_shared_decode", 3, None)])
def test_ep_shards_sum_to_the_whole_layer(moe, name, n, n_sample):
    lay = SyntheticLayer(CONFIGS[name], 2)
    c = lay.cfg
    sample = (np.arange(c.tokens) if n_sample is None else
              np.sort(np.random.default_rng(7).choice(c.tokens, n_sample, replace=False)))
    say("ep shards", name, "seed 2, n", n, "tokens", len(sample))
    total, idx = run_shards(moe, lay, n, sample)
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    exp_idx, _ = expected_routing(lg_ref, idx, c.top_k)
    np.testing.assert_array_equal(idx, exp_idx)
    ref = oracle.layer_forward_synthetic(lay, idx=exp_idx, sample=sample, offloaded=True)
    want = ref["out_res"] + ref["out_off"]
    err = rel_l2(total, want)
    say(f"  rel-L2 {err:.3e} (tol {TOL[c.dtype]})")
    assert err <= TOL[c.dtype]


def test_ep_shards_with_empty_shards(moe):
    """Fewer experts and shared columns than shards: some shards hold nothing and add zeros."""
    lay = make_layer(9, 64, 4, 64, 2, dtype="bf16", shared=1, shared_ffn=128, n_resident=2, residency="random",
                     bias="zipf", seed=4)
    say("ep shards, 4 experts and 2 shared units over 8 shards")
    sample = np.arange(9)
    total, idx = run_shards(moe, lay, 8, sample)
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    exp_idx, _ = expected_routing(lg_ref, idx, 2)
    ref = oracle.layer_forward_synthetic(lay, idx=exp_idx, sample=sample, offloaded=True)
    err = rel_l2(total, ref["out_res"] + ref["out_off"])
    say(f"  rel-L2 {err:.3e} (tol {TOL['bf16']})")
    assert err <= TOL["bf16"]
