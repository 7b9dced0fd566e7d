"""Bookkeeping baseline (per-expert mask -> gather -> FFN launch -> scatter-add) vs the
oracle and vs the fused, repacked layer forward (SAEM Section IV-E.1 A/B).

Both paths use the library's router and FFN kernels; the baseline's output must
be the same resident partial layer output (the scatter-add is atomic, so only a
float tolerance applies between the two paths)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_support import DELTA, TOL, expected_routing, host_f64, rel_l2
from workloads import CONFIGS, SyntheticLayer

pytestmark = pytest.mark.gpu


def say(*a):
    print("[bookkeeping]", *a, flush=True)


@pytest.mark.parametrize("name", ["c2_mixtral_decode", "c3_shared_decode", "c6_qwen3_decode"])
def test_bookkeeping_matches_oracle_and_fused(name):
    from paper_2608_21614_amd import MOE_F32
    from paper_2608_21614_amd.bookkeeping import BookkeepingLayer
    from paper_2608_21614_amd.device import DeviceLayer, to_host
    say(name)
    lay = SyntheticLayer(CONFIGS[name], 0)
    c = lay.cfg
    dev = DeviceLayer(lay)
    bk = BookkeepingLayer(dev)
    out_bk = bk.forward()
    o = dev.alloc_outputs(out_dtype=MOE_F32)
    dev.forward(o)
    torch.cuda.synchronize()
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    lg = to_host(bk.o["logits"]).astype(np.float64)
    assert np.abs(lg - lg_ref).max() < DELTA / 2
    idx = to_host(bk.o["topk_idx"])
    exp_idx, _ = expected_routing(lg_ref, idx, c.top_k)
    np.testing.assert_array_equal(idx, exp_idx)
    np.testing.assert_array_equal(idx, to_host(o["topk_idx"]))
    sample = np.arange(0, c.tokens, max(1, c.tokens // 16))
    ref = oracle.layer_forward_synthetic(lay, idx=exp_idx, sample=sample, offloaded=False)
    err = rel_l2(host_f64(out_bk)[ref["sample"]], ref["out_res"])
    err_ab = rel_l2(host_f64(out_bk), host_f64(o["out"]))
    say(f"  vs oracle {err:.3e}, vs fused {err_ab:.3e}, host syncs {bk.last['host_syncs']}")
    assert err <= TOL["bf16"]
    assert err_ab <= TOL["bf16"]
