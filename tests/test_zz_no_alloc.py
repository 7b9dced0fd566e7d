"""moe_layer_forward_noalloc (the fused forward on the library's fixed per-GPU
scratch array) against moe_layer_forward with a caller workspace, through the C
ABI: identical outputs, bit for bit, on two calls in a row -- the second with a
smaller batch of another layer, so it runs on whatever the first call left in
the array.  Then a layer too large for the array is refused before anything runs.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

from workloads import CONFIGS, SyntheticLayer, make_layer

pytestmark = pytest.mark.gpu


def say(*a):
    print("[noalloc]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def moe():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_21614_amd as m
    return m


OUT_KEYS = ("out", "logits", "topk_idx", "topk_w", "counts", "seg_start", "perm", "inv_perm", "n_res", "off_rows",
            "off_w")


def _both(moe, lay):
    from paper_2608_21614_amd.device import DeviceLayer
    dev = DeviceLayer(lay)
    ref, got = dev.alloc_outputs(), dev.alloc_outputs()
    for o in (ref, got):        # different garbage in every output: nothing may be left unwritten
        for key in OUT_KEYS:
            o[key].fill_(3 if o is ref else 5)
    moe.moe_layer_forward(dev.args(ref), dev.ws)
    moe.moe_layer_forward_noalloc(dev.args(got))
    torch.cuda.synchronize()
    return dev, ref, got


def _check_equal(lay, ref, got):
    c = lay.cfg
    P = c.tokens * c.top_k
    n_res = int(ref["n_res"][0].item())
    for key in ("out", "logits", "topk_idx", "topk_w", "counts", "seg_start", "n_res"):
        assert torch.equal(ref[key], got[key]), key
    for key in ("perm", "inv_perm"):
        assert torch.equal(ref[key][:P], got[key][:P]), key
    # the offloaded list: its P - n_res rows
    assert torch.equal(ref["off_rows"][: P - n_res], got["off_rows"][: P - n_res])
    assert torch.equal(ref["off_w"][: P - n_res], got["off_w"][: P - n_res])


@pytest.mark.parametrize("first,second", [
    ("c3_shared_decode", "small"),
    ("c2_mixtral_decode", "c1_tiny_f32"),
])
def test_noalloc_equals_workspace_forward_two_calls(moe, first, second):
    layers = [SyntheticLayer(CONFIGS[first], 2)]
    if second == "small":
        layers.append(make_layer(9, 256, 60, 128, 4, dtype="bf16", shared=1, shared_ffn=64, n_resident=20,
                                 residency="random", bias="zipf", seed=7))
    else:
        layers.append(SyntheticLayer(CONFIGS[second], 3))
    assert layers[1].cfg.tokens < layers[0].cfg.tokens
    for i, lay in enumerate(layers):
        c = lay.cfg
        say(f"call {i}: {c.name} T={c.tokens} H={c.hidden} E={c.experts} F={c.ffn} k={c.top_k} S={c.shared}")
        dims = moe.make_dims(c.tokens, c.hidden, c.experts, c.ffn, c.top_k, c.shared, c.shared_ffn,
                             int(lay.resident.sum()), moe.MOE_BF16 if c.dtype == "bf16" else moe.MOE_F32)
        assert moe.moe_workspace_bytes(dims) <= moe.MOE_NOALLOC_SCRATCH_BYTES
        dev, ref, got = _both(moe, lay)
        _check_equal(lay, ref, got)
        say(f"call {i}: identical outputs")
        del dev, ref, got


def test_noalloc_refuses_a_layer_above_the_limit(moe):
    from paper_2608_21614_amd.device import DeviceLayer
    say("c4_prefill: workspace above the scratch limit")
    lay = make_layer(2048, 128, 64, 64, 6, dtype="bf16", shared=2, shared_ffn=4096, n_resident=48, seed=1)
    dev = DeviceLayer(lay)
    assert moe.moe_workspace_bytes(dev.dims) > moe.MOE_NOALLOC_SCRATCH_BYTES
    o = dev.alloc_outputs()
    o["out"].fill_(9)
    with pytest.raises(moe.MoeError) as ei:
        moe.moe_layer_forward_noalloc(dev.args(o))
    assert ei.value.status == moe.MOE_ERR_SCRATCH_LIMIT
    torch.cuda.synchronize()
    assert bool((o["out"] == 9).all())     # nothing ran
