"""The expert-parallel split of a layer (``workloads.ExpertShard``), checked on the CPU.

Under n-way expert parallelism every GPU routes the whole batch and runs the
experts it holds; the layer's output is the sum of the GPUs' partial outputs
(Section II-A: the output is a gate-weighted sum over the selected experts plus
the shared experts, and a SwiGLU expert's output is a sum over its FFN columns).
These tests pin the split itself: the shards partition the experts and the
shared columns, and the oracle run on each shard, summed, gives the oracle's
whole-layer output.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from workloads import CONFIGS, ExpertShard, SyntheticLayer, make_layer


@pytest.mark.parametrize("name", ["c2_mixtral_decode", "c3_shared_decode", "c4_prefill", "c6_qwen3_decode"])
@pytest.mark.parametrize("n", [1, 2, 8])
def test_shards_partition_experts_and_shared_columns(name, n):
    lay = SyntheticLayer(CONFIGS[name], 0)
    c = lay.cfg
    shards = [ExpertShard(lay, n, g) for g in range(n)]
    held = np.concatenate([s.expert_ids for s in shards])
    np.testing.assert_array_equal(np.sort(held), np.arange(c.experts))   # every expert exactly once
    for s in shards:
        assert (np.diff(s.expert_ids) == 1).all()                       # a contiguous id block
        np.testing.assert_array_equal(s.expert_slot[s.expert_ids], np.arange(s.n_slots))
        assert (s.expert_slot[~s.resident] == -1).all()
        assert s.cfg.shared_ffn % 64 == 0
        assert s.x is lay.x and s.w_router is lay.w_router and s.bias is lay.bias
    if c.shared:
        cols = [s.shared_cols for s in shards]
        assert cols[0][0] == 0 and cols[-1][1] == c.shared_ffn
        assert all(a[1] == b[0] for a, b in zip(cols, cols[1:]))        # adjacent, no gap, no overlap
        assert max(f1 - f0 for f0, f1 in cols) - min(f1 - f0 for f0, f1 in cols) <= 64
    sizes = [s.n_slots for s in shards]
    assert max(sizes) - min(sizes) <= 1


def test_shard_shared_slices_are_the_layers_columns():
    lay = make_layer(4, 64, 4, 64, 2, shared=2, shared_ffn=320, seed=3)
    F = 320
    for g in range(3):
        s = ExpertShard(lay, 3, g)
        f0, f1 = s.shared_cols
        for e in range(2):
            w13, w2 = s.ws13(e), s.ws2(e)
            assert w13.shape == (2 * (f1 - f0), 64) and w2.shape == (64, f1 - f0)
            np.testing.assert_array_equal(w13[: f1 - f0], lay.ws13(e)[f0:f1])          # gate rows
            np.testing.assert_array_equal(w13[f1 - f0:], lay.ws13(e)[F + f0:F + f1])   # up rows
            np.testing.assert_array_equal(w2, lay.ws2(e)[:, f0:f1])


@pytest.mark.parametrize("T,H,E,F,k,S,Fs,n,dtype", [
    (24, 128, 20, 128, 4, 2, 320, 8, "bf16"),   # 5 shared units over 8 shards: three shards hold no shared expert
    (9, 64, 4, 64, 2, 1, 128, 8, "f32"),        # fewer experts than shards: four shards hold nothing routed
    (16, 64, 8, 192, 2, 0, 0, 3, "f32"),        # uneven blocks (3, 3, 2)
])
def test_oracle_over_shards_sums_to_the_whole_layer(T, H, E, F, k, S, Fs, n, dtype):
    lay = make_layer(T, H, E, F, k, dtype=dtype, shared=S, shared_ffn=Fs, n_resident=E // 2, residency="random",
                     bias="zipf", seed=T + E)
    whole = oracle.layer_forward_synthetic(lay, offloaded=True)
    full = whole["out_res"] + whole["out_off"]
    total = np.zeros_like(full)
    for g in range(n):
        part = oracle.layer_forward_synthetic(ExpertShard(lay, n, g), offloaded=False)
        np.testing.assert_array_equal(part["idx"], whole["idx"])         # routing is replicated
        assert not part["out_off"].any()
        total += part["out_res"]
    scale = np.abs(full).max()
    assert scale > 0
    np.testing.assert_allclose(total, full, rtol=0, atol=1e-12 * scale)


def test_shard_rejects_bad_index():
    lay = make_layer(4, 64, 4, 64, 2, seed=1)
    with pytest.raises(ValueError):
        ExpertShard(lay, 2, 2)
    with pytest.raises(ValueError):
        ExpertShard(lay, 0, 0)
