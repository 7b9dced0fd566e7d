"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Every test prints the case it runs (config, seed, shape) before touching the
GPU.  Inputs come from the seeded generators in ``workloads``; expected values
from ``oracle`` only.
"""
from __future__ import annotations

import sys

import numpy as np
import pytest
import torch

import oracle
from gpu_support import (DELTA, LOGIT_TOL, TOL, check_offloaded_list, expected_routing, host_f64,
                         rel_l2, row_rel_l2)
from workloads import CONFIGS, SyntheticLayer, bf16_bits_to_f32, make_layer

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


def _dev(a):
    from paper_2608_21614_amd.device import to_device
    return to_device(a)


def _host(t):
    from paper_2608_21614_amd.device import to_host
    return to_host(t)


def x_as_f32(layer):
    return bf16_bits_to_f32(layer.x) if layer.cfg.dtype == "bf16" else layer.x


# ---------------------------------------------------------------------------
# weight packing into the tile layout
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("rows,cols,dtype", [(16, 32, "bf16"), (2816, 2048, "bf16"), (64, 1408, "bf16"),
                                            (128, 256, "f32"), (48, 96, "f32")])
def test_pack_weights_layout(moe, rows, cols, dtype):
    """Packed element 8*l + i of block (rt, s) is W[16 rt + l%16][32 s + 8 (l/16) + i]; the inverse recovers W."""
    say("pack", rows, cols, dtype)
    rng = np.random.default_rng(rows + cols)
    w = rng.integers(0, 1 << 16, size=(rows, cols), dtype=np.uint16) if dtype == "bf16" else \
        rng.standard_normal((rows, cols)).astype(np.float32)
    src = _dev(w)
    dst = torch.empty_like(src)
    moe.moe_pack_weights(src, dst)
    torch.cuda.synchronize()
    got = _host(dst).reshape(rows // 16, cols // 32, 4, 16, 8)
    back = got.transpose(0, 3, 1, 2, 4).reshape(rows, cols)
    np.testing.assert_array_equal(back, w)
    # one explicit element
    rt, s_, l, i = rows // 16 - 1, cols // 32 - 1, 37, 5
    assert _host(dst).reshape(-1)[(rt * (cols // 32) + s_) * 512 + 8 * l + i] == w[16 * rt + l % 16, 32 * s_ + 8 * (l // 16) + i]


# ---------------------------------------------------------------------------
# routing on given scores: bit-exact selection
# ---------------------------------------------------------------------------

def _constructed_logits(T, E, rng):
    lg = rng.standard_normal((T, E)).astype(np.float32)
    lg[0] = 0.0                                   # all equal
    if T > 1:
        lg[1] = -np.inf                           # all -inf
    if T > 2:
        lg[2] = np.round(lg[2])                   # many exact ties
    if T > 3:
        lg[3, : min(E, 3)] = 7.0                  # tie at the top
    if T > 4:
        lg[4] = np.where(rng.random(E) < 0.5, -np.inf, lg[4])
    if T > 5:
        lg[5] = -0.0
        lg[5, E // 2] = 0.0                       # -0 == +0
    lg[6:] = np.round(lg[6:] * 4) / 4            # coarse values: frequent ties
    return lg


@pytest.mark.parametrize("T,E,k", [(7, 1, 1), (33, 8, 2), (64, 60, 4), (100, 64, 6), (40, 128, 8), (70, 256, 8),
                                   (17, 256, 1), (20, 8, 8), (1, 5, 3)])
def test_route_topk_given_scores_bit_exact(moe, T, E, k):
    say("route given scores", T, E, k)
    rng = np.random.default_rng(T * 31 + E + k)
    lg = _constructed_logits(T, E, rng)
    dims = moe.make_dims(T, 64, E, 64, k, slots=0)
    d_lg = _dev(lg)
    d_idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
    d_w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(moe.moe_workspace_bytes(dims), dtype=torch.uint8, device="cuda")
    moe.moe_route_topk(dims, None, None, None, d_lg, d_idx, d_w, ws, logits_in=True)
    torch.cuda.synchronize()
    ref_idx, ref_w = oracle.topk(lg.astype(np.float64), k)
    np.testing.assert_array_equal(_host(d_idx), ref_idx)
    np.testing.assert_allclose(_host(d_w), ref_w, rtol=2e-6, atol=1e-7)
    np.testing.assert_array_equal(_host(d_lg), lg)  # scores untouched


# ---------------------------------------------------------------------------
# routing on computed scores
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,T,H,E,k,bias", [
    ("bf16", 1, 64, 8, 2, "none"), ("bf16", 17, 256, 60, 4, "zipf"), ("bf16", 100, 2048, 64, 6, "zipf"),
    ("bf16", 33, 4096, 8, 2, "none"), ("bf16", 16, 128, 256, 8, "zipf"), ("f32", 16, 256, 8, 2, "none"),
    ("f32", 21, 64, 130, 5, "zipf"), ("f32", 100, 256, 64, 6, "zipf"),
])
def test_route_topk_computed_scores(moe, dtype, T, H, E, k, bias):
    say("route computed", dtype, T, H, E, k, bias)
    lay = make_layer(T, H, E, 64, k, dtype=dtype, bias=bias, n_resident=E // 2, residency="random", seed=T + E)
    dims = moe.make_dims(T, H, E, 64, k, slots=0, dtype=1 if dtype == "bf16" else 0)
    d_lg = torch.empty((T, E), dtype=torch.float32, device="cuda")
    d_idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
    d_w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(moe.moe_workspace_bytes(dims), dtype=torch.uint8, device="cuda")
    moe.moe_route_topk(dims, _dev(lay.x), _dev(lay.w_router), None if lay.bias is None else _dev(lay.bias),
                       d_lg, d_idx, d_w, ws)
    torch.cuda.synchronize()
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    lg = _host(d_lg).astype(np.float64)
    assert np.abs(lg - lg_ref).max() < DELTA / 2
    idx = _host(d_idx)
    exp_idx, _ = expected_routing(lg_ref, idx, k)
    np.testing.assert_array_equal(idx, exp_idx)
    # the GPU's gate is the softmax of its own scores over its selection
    np.testing.assert_allclose(_host(d_w), oracle.gate_weights(lg, idx), rtol=2e-6, atol=1e-7)


# ---------------------------------------------------------------------------
# repacking
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T,E,k,mode", [(1, 1, 1, "all"), (4, 4, 2, "paper"), (32, 8, 2, "random"),
                                         (64, 60, 4, "random"), (2048, 64, 6, "random"), (3000, 256, 8, "random"),
                                         (500, 16, 3, "none"), (257, 64, 6, "all"), (40, 8, 2, "invalid"),
                                         # 128 chunks of 1024 pairs (one per workgroup), then 157 (two per
                                         # workgroup for some)
                                         (16384, 128, 8, "all"), (20000, 64, 8, "random")])
def test_repack_bit_exact(moe, T, E, k, mode):
    say("repack", T, E, k, mode)
    rng = np.random.default_rng(T + E * 7 + k)
    if mode == "paper":
        idx = np.array([[0, 2], [1, 2], [1, 3], [0, 2]], dtype=np.int32)
    else:
        idx = np.stack([rng.choice(E, k, replace=False) for _ in range(T)]).astype(np.int32)
        # Zipf-like skew: pull many pairs onto a few experts
        hot = rng.random((T, 1)) < 0.6
        idx[:, :1] = np.where(hot, rng.integers(0, min(E, 3), (T, 1)), idx[:, :1])
        idx = np.stack([row if len(set(row)) == k else rng.choice(E, k, replace=False) for row in idx]).astype(np.int32)
    res = {"all": np.ones(E, bool), "none": np.zeros(E, bool)}.get(mode, rng.random(E) < 0.5)
    if mode == "paper":
        res = np.array([1, 0, 1, 0], bool)
    slot = np.full(E, -1, np.int32)
    slot[res] = rng.permutation(int(res.sum()))
    if mode == "random" and E > 4:
        slot[np.flatnonzero(~res)[:1]] = 10_000   # out-of-range slot: offloaded
    if mode == "invalid":
        idx[3, 0] = E + 5
        idx[7, 1] = -1
    slots = int(res.sum())
    dims = moe.make_dims(T, 64, E, 64, k, slots=slots)
    P = T * k
    out = {n: torch.full((max(P, 1),), -7, dtype=torch.int32, device="cuda") for n in ("perm", "inv")}
    counts = torch.empty(E, dtype=torch.int32, device="cuda")
    seg = torch.empty(E, dtype=torch.int32, device="cuda")
    nres = torch.empty(1, dtype=torch.int32, device="cuda")
    moe.moe_repack(dims, _dev(idx), None, _dev(slot), None, counts, seg, out["perm"], out["inv"], nres)
    torch.cuda.synchronize()
    eff_res = (slot >= 0) & (slot < slots)
    if mode == "invalid":
        valid = (idx >= 0) & (idx < E)
        assert _host(counts).sum() == valid.sum()
        np.testing.assert_array_equal(_host(counts), np.bincount(idx[valid], minlength=E))
        inv = _host(out["inv"])
        assert inv[3 * k] == -1 and inv[7 * k + 1] == -1
        # the packed rows left over by the two dropped pairs hold no pair
        perm = _host(out["perm"])
        n_valid = int(valid.sum())
        np.testing.assert_array_equal(perm[n_valid:P], -1)
        assert sorted(perm[:n_valid].tolist()) == sorted(np.flatnonzero(valid.reshape(-1)).tolist())
        return
    ref = oracle.repack(idx, eff_res)
    np.testing.assert_array_equal(_host(counts), ref["counts"])
    np.testing.assert_array_equal(_host(seg), ref["seg_start"])
    np.testing.assert_array_equal(_host(out["perm"])[:P], ref["perm"])
    np.testing.assert_array_equal(_host(out["inv"])[:P], ref["inv_perm"])
    assert int(_host(nres)[0]) == ref["n_res"]


def test_offload_pack_bit_exact(moe):
    say("offload pack c3-like")
    lay = make_layer(64, 2048, 60, 64, 4, dtype="bf16", n_resident=30, residency="random", bias="zipf", seed=5)
    T, E, k, H = 64, 60, 4, 2048
    dims = moe.make_dims(T, H, E, 64, k, slots=30)
    d_lg = torch.empty((T, E), dtype=torch.float32, device="cuda")
    d_idx = torch.empty((T, k), dtype=torch.int32, device="cuda")
    d_w = torch.empty((T, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(moe.moe_workspace_bytes(dims), dtype=torch.uint8, device="cuda")
    moe.moe_route_topk(dims, _dev(lay.x), _dev(lay.w_router), _dev(lay.bias), d_lg, d_idx, d_w, ws)
    counts = torch.empty(E, dtype=torch.int32, device="cuda")
    seg = torch.empty(E, dtype=torch.int32, device="cuda")
    perm = torch.empty(T * k, dtype=torch.int32, device="cuda")
    inv = torch.empty(T * k, dtype=torch.int32, device="cuda")
    nres = torch.empty(1, dtype=torch.int32, device="cuda")
    off_rows = torch.zeros((T * k, H), dtype=torch.bfloat16, device="cuda")
    off_w = torch.zeros(T * k, dtype=torch.float32, device="cuda")
    moe.moe_repack(dims, d_idx, d_w, _dev(lay.expert_slot), _dev(lay.x), counts, seg, perm, inv, nres, off_rows, off_w)
    torch.cuda.synchronize()
    n_res = int(_host(nres)[0])
    assert n_res < T * k  # this seed has offloaded pairs
    check_offloaded_list(lay.x, k, _host(perm), n_res, _host(off_rows), _host(off_w), _host(d_w))


# ---------------------------------------------------------------------------
# fused layer forward
# ---------------------------------------------------------------------------

def run_and_check_layer(moe, lay, sample=None, check_off=True, offloaded_oracle=False):
    """Fused forward on the GPU vs the oracle; returns (device outputs, oracle result)."""
    from paper_2608_21614_amd.device import DeviceLayer
    c = lay.cfg
    T, E, k, H = c.tokens, c.experts, c.top_k, c.hidden
    dev = DeviceLayer(lay)
    o = dev.alloc_outputs()
    dev.forward(o)
    torch.cuda.synchronize()
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    lg = _host(o["logits"]).astype(np.float64)
    idx = _host(o["topk_idx"])
    if T:
        assert np.abs(lg - lg_ref).max() < DELTA / 2, "router scores off by more than DELTA/2"
        err_lg = rel_l2(lg, lg_ref)
        say(f"  logits rel-L2 {err_lg:.3e} (tol {LOGIT_TOL})")
        assert err_lg <= LOGIT_TOL
        # given identical scores (the GPU's own fp32 logits), routing is bit-exact
        own_idx, own_w = oracle.topk(lg, k)
        np.testing.assert_array_equal(idx, own_idx)
        np.testing.assert_allclose(_host(o["topk_w"]), own_w, rtol=2e-6, atol=1e-7)
    exp_idx, _ = expected_routing(lg_ref, idx, k) if T else (idx, {})
    np.testing.assert_array_equal(idx, exp_idx)
    ref = oracle.layer_forward_synthetic(lay, idx=exp_idx, sample=sample, offloaded=offloaded_oracle)
    np.testing.assert_array_equal(_host(o["counts"]), ref["counts"])
    np.testing.assert_array_equal(_host(o["seg_start"]), ref["seg_start"])
    P = T * k
    np.testing.assert_array_equal(_host(o["perm"])[:P], ref["perm"])
    np.testing.assert_array_equal(_host(o["inv_perm"])[:P], ref["inv_perm"])
    n_res = int(_host(o["n_res"])[0])
    assert n_res == ref["n_res"]
    if T:
        np.testing.assert_allclose(_host(o["topk_w"]), ref["w"], rtol=5e-5, atol=1e-6)
        out = host_f64(o["out"])[ref["sample"]]
        err = rel_l2(out, ref["out_res"])
        say(f"  rel-L2 {err:.3e} (tol {TOL[c.dtype]})")
        assert err <= TOL[c.dtype]
        if check_off:
            check_offloaded_list(lay.x, k, _host(o["perm"])[:P], n_res, _host(o["off_rows"]), _host(o["off_w"]),
                                 _host(o["topk_w"]))
    return dev, o, ref


@pytest.mark.parametrize("seed", range(5))
def test_layer_c1_tiny_f32(moe, seed):
    say("layer c1_tiny_f32 seed", seed)
    run_and_check_layer(moe, SyntheticLayer(CONFIGS["c1_tiny_f32"], seed))


@pytest.mark.parametrize("seed", range(5))
def test_layer_c2_mixtral_decode(moe, seed):
    say("layer c2_mixtral_decode seed", seed)
    run_and_check_layer(moe, SyntheticLayer(CONFIGS["c2_mixtral_decode"], seed))


@pytest.mark.parametrize("seed", range(5))
def test_layer_c3_shared_decode(moe, seed):
    say("layer c3_shared_decode seed", seed)
    run_and_check_layer(moe, SyntheticLayer(CONFIGS["c3_shared_decode"], seed))


@pytest.mark.parametrize("seed", range(5))
def test_layer_c6_qwen3_decode(moe, seed):
    say("layer c6_qwen3_decode seed", seed)
    run_and_check_layer(moe, SyntheticLayer(CONFIGS["c6_qwen3_decode"], seed))


def test_layer_calls_share_one_workspace(moe):
    """Decode calls of two different layers alternate on one workspace that starts
    filled with garbage: every call's routing and repack match its own oracle (no
    state carries over between calls through the workspace)."""
    from paper_2608_21614_amd.device import DeviceLayer
    lays = [make_layer(48, 256, 60, 128, 4, dtype="bf16", shared=1, shared_ffn=128, n_resident=30,
                       residency="random", bias="zipf", seed=s) for s in (21, 22)]
    devs = [DeviceLayer(l) for l in lays]
    ws = torch.full_like(devs[0].ws, 0x5A)
    outs = [d.alloc_outputs() for d in devs]
    for it in range(3):
        for lay, dev, o in zip(lays, devs, outs):
            say("shared workspace: call", it, "seed", lay.seed)
            dev.ws = ws
            dev.forward(o)
            torch.cuda.synchronize()
            lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
            idx = _host(o["topk_idx"])
            exp_idx, _ = expected_routing(lg_ref, idx, lay.cfg.top_k)
            np.testing.assert_array_equal(idx, exp_idx)
            ref = oracle.repack(exp_idx, lay.resident)
            np.testing.assert_array_equal(_host(o["counts"]), ref["counts"])
            np.testing.assert_array_equal(_host(o["perm"]), ref["perm"])
            np.testing.assert_array_equal(_host(o["inv_perm"]), ref["inv_perm"])
            assert int(_host(o["n_res"])[0]) == ref["n_res"]


def check_ffn_rows(moe, dev, lay, ref):
    """The grouped FFN's rows (moe_grouped_ffn, the same kernels as the fused call) against the
    oracle's expert outputs: every resident packed row, and every shared-expert row."""
    c = lay.cfg
    T, k, H, S = c.tokens, c.top_k, c.hidden, c.shared
    o, y, _ = _standalone_chain(moe, dev)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_host(o["perm"])[: T * k], ref["perm"])
    n_res = ref["n_res"]
    yr = _host(y)
    got, want = yr[:n_res], ref["y_rows"][:n_res]
    err, worst = rel_l2(got, want), float(row_rel_l2(got, want).max()) if n_res else 0.0
    say(f"  FFN rows: {n_res} resident rows rel-L2 {err:.3e}, worst row {worst:.3e}")
    assert err <= TOL[c.dtype] and worst <= TOL[c.dtype]
    toks = np.arange(T, dtype=np.int32)
    for s_ in range(S):
        want = oracle.expert_ffn(lay.x, toks, lay.ws13(s_), lay.ws2(s_))
        got = yr[T * k + s_ * T: T * k + (s_ + 1) * T]
        err, worst = rel_l2(got, want), float(row_rel_l2(got, want).max())
        say(f"  FFN rows: shared expert {s_} rel-L2 {err:.3e}, worst row {worst:.3e}")
        assert err <= TOL[c.dtype] and worst <= TOL[c.dtype]


@pytest.mark.parametrize("seed", range(5))
def test_layer_c4_prefill(moe, seed):
    """The prefill config at full size: every token's output, and every FFN row."""
    say("layer c4_prefill seed", seed, "(all 2048 tokens, all FFN rows)")
    lay = SyntheticLayer(CONFIGS["c4_prefill"], seed)
    dev, _, ref = run_and_check_layer(moe, lay)
    check_ffn_rows(moe, dev, lay, ref)


def test_layer_c4_prefill_f32(moe):
    """The prefill shape in fp32 (the fp32 MFMA path at full size): every token's output at
    the fp32 bar, and every FFN row."""
    say("layer c4_prefill_f32 seed 0 (all 2048 tokens, all FFN rows)")
    lay = SyntheticLayer(CONFIGS["c4_prefill_f32"], 0)
    dev, _, ref = run_and_check_layer(moe, lay)
    check_ffn_rows(moe, dev, lay, ref)


@pytest.mark.parametrize("name", ["c2_mixtral_decode", "c3_shared_decode"])
def test_ffn_rows_decode(moe, name):
    """Decode configs: every resident packed row and shared row of the grouped FFN (split-K sums added)."""
    from paper_2608_21614_amd.device import DeviceLayer
    say("FFN rows", name, "seed 1")
    lay = SyntheticLayer(CONFIGS[name], 1)
    dev, _, ref = run_and_check_layer(moe, lay)
    check_ffn_rows(moe, dev, lay, ref)


def test_layer_prefill_all_256_experts_active(moe):
    """A prefill batch whose 256 experts are all resident and all receive tokens: the tiled
    kernel's per-expert tile list then holds 256 groups (its end entry past the last lane's)."""
    say("layer prefill, 256 experts all resident and active")
    lay = make_layer(400, 64, 256, 64, 8, dtype="bf16", n_resident=256, residency="random", bias="none", seed=11)
    dev, o, ref = run_and_check_layer(moe, lay)
    assert (ref["counts"] > 0).all(), "every expert must be active for this case"
    check_ffn_rows(moe, dev, lay, ref)


EDGE = [
    # (T, H, E, F, k, S, Fs, dtype, resident)
    (0, 64, 8, 64, 2, 0, 0, "bf16", 4),
    (1, 64, 1, 64, 1, 0, 0, "bf16", 1),
    (7, 128, 8, 192, 2, 1, 64, "bf16", 3),
    (16, 256, 8, 512, 8, 0, 0, "bf16", 8),
    (63, 256, 60, 1408, 4, 1, 320, "bf16", 30),
    (64, 64, 64, 64, 6, 2, 128, "bf16", 0),
    (65, 128, 16, 128, 2, 0, 0, "bf16", 16),
    (130, 192, 64, 1408, 6, 2, 128, "bf16", 48),
    (33, 128, 256, 64, 8, 0, 0, "bf16", 100),
    (20, 64, 128, 128, 8, 1, 64, "f32", 64),
    (9, 64, 4, 64, 4, 2, 128, "f32", 0),
    (100, 64, 8, 128, 2, 1, 64, "f32", 4),
    (2, 4096, 8, 14336, 2, 0, 0, "bf16", 4),
    # a prefill batch one token past a 2048 multiple: the last 256-token tile, the last
    # 8-token router workgroup and the last 1024-pair repack chunk are all ragged
    (2049, 128, 64, 192, 6, 1, 64, "bf16", 40),
    (2049, 64, 8, 64, 2, 0, 0, "f32", 6),
    # the ABI's limits at once: 256 experts, top-8, eight shared experts
    (40, 128, 256, 64, 8, 8, 64, "bf16", 256),
    (200, 128, 256, 64, 8, 8, 128, "bf16", 128),
    (24, 64, 16, 64, 8, 8, 64, "f32", 8),
    # fp32 prefill on MFMA: groups of several 64-row chunks (one ragged), shared
    # experts wider than the routed ones, and more experts than resident slots
    (300, 256, 16, 192, 4, 2, 320, "f32", 10),
    (65, 128, 4, 64, 1, 1, 64, "f32", 4),
]


@pytest.mark.parametrize("T,H,E,F,k,S,Fs,dtype,res", EDGE)
def test_layer_edge_shapes(moe, T, H, E, F, k, S, Fs, dtype, res):
    say("layer edge", T, H, E, F, k, S, Fs, dtype, res)
    lay = make_layer(T, H, E, F, k, dtype=dtype, shared=S, shared_ffn=Fs, n_resident=res, residency="random",
                     bias="zipf", seed=T * 3 + E)
    run_and_check_layer(moe, lay)


@pytest.mark.parametrize("T,H,E,F,k,S,Fs,dtype,res", [
    (8, 128, 64, 192, 4, 0, 0, "bf16", 32),    # T k = slots: routed items map to slots
    (4, 64, 32, 128, 8, 1, 64, "bf16", 32),    # every expert resident, most slots idle
    (16, 128, 64, 128, 4, 0, 0, "f32", 64),    # E = slots = T k
    (2, 128, 64, 192, 4, 1, 64, "bf16", 16),   # T k < slots: items follow the active list
    (3, 64, 40, 64, 5, 0, 0, "f32", 20),       # T k < slots, fp32
])
def test_layer_decode_slot_mapping(moe, T, H, E, F, k, S, Fs, dtype, res):
    """The fused decode forward maps routed items to residency slots when every slot can
    hold an active expert (T k >= slots), and to the active list otherwise; slots whose
    expert gets no token exit.  Both mappings, at the layer bar, over two seeds."""
    for seed in (0, 1):
        say("layer decode, slot mapping", T, H, E, F, k, S, Fs, dtype, res, "seed", seed)
        lay = make_layer(T, H, E, F, k, dtype=dtype, shared=S, shared_ffn=Fs, n_resident=res, residency="random",
                         bias="zipf", seed=seed + 5 * T + E)
        run_and_check_layer(moe, lay)


@pytest.mark.parametrize("T,H,E,F,k,S,Fs,dtype,res", [
    (4, 64, 200, 704, 7, 0, 0, "f32", 66),
    (4, 64, 200, 704, 7, 2, 64, "f32", 66),
    (9, 64, 60, 1408, 4, 1, 320, "bf16", 30),
    (40, 128, 16, 192, 2, 2, 64, "bf16", 8),
    (17, 64, 8, 64, 2, 0, 0, "f32", 4),
])
def test_layer_decode_few_k_steps_repeated(moe, T, H, E, F, k, S, Fs, dtype, res):
    """Decode layers whose K (H = 64 or 128) gives some waves of the stream kernel no K
    steps: those waves reach the epilogue first.  Ten calls of each, every one at the bar
    (the FFN's prologue data must not share LDS with the epilogue's partial tiles)."""
    from paper_2608_21614_amd.device import DeviceLayer
    say("layer decode, few K steps, ten calls", T, H, E, F, k, S, Fs, dtype, res)
    lay = make_layer(T, H, E, F, k, dtype=dtype, shared=S, shared_ffn=Fs, n_resident=res, residency="random",
                     bias="zipf", seed=474)
    dev, o, ref = run_and_check_layer(moe, lay)
    first = host_f64(o["out"])
    for _ in range(9):
        o["out"].zero_()
        dev.forward(o)
        torch.cuda.synchronize()
        got = host_f64(o["out"])
        np.testing.assert_array_equal(got, first)  # deterministic, and every call complete
        err = rel_l2(got[ref["sample"]], ref["out_res"])
        assert err <= TOL[dtype]


def test_layer_logits_in_routes_given_scores(moe):
    """MOE_LOGITS_IN: the fused forward routes caller scores, including exact ties, bit-exactly."""
    from paper_2608_21614_amd.device import DeviceLayer
    say("layer logits-in c3-like")
    lay = make_layer(64, 256, 60, 128, 4, dtype="bf16", shared=1, shared_ffn=128, n_resident=30,
                     residency="random", seed=9)
    dev = DeviceLayer(lay)
    o = dev.alloc_outputs()
    rng = np.random.default_rng(9)
    lg = np.round(rng.standard_normal((64, 60)) * 2).astype(np.float32)  # integers: many ties
    o["logits"].copy_(_dev(lg))
    dev.forward(o, logits_in=True)
    torch.cuda.synchronize()
    ref = oracle.layer_forward_synthetic(lay, logits=lg.astype(np.float64), offloaded=False)
    np.testing.assert_array_equal(_host(o["topk_idx"]), ref["idx"])
    np.testing.assert_array_equal(_host(o["perm"]), ref["perm"])
    assert rel_l2(host_f64(o["out"]), ref["out_res"]) <= TOL["bf16"]


# ---------------------------------------------------------------------------
# determinism, standalone chain, host merge
# ---------------------------------------------------------------------------

def _standalone_chain(moe, dev, y_off=None):
    """route -> repack -> grouped_ffn -> combine through the four separate entry points."""
    c = dev.cfg
    T, E, k, H, S = c.tokens, c.experts, c.top_k, c.hidden, c.shared
    o = dev.alloc_outputs()
    moe.moe_route_topk(dev.dims, dev.x, dev.w_router, dev.bias, o["logits"], o["topk_idx"], o["topk_w"], dev.ws)
    moe.moe_repack(dev.dims, o["topk_idx"], o["topk_w"], dev.expert_slot, dev.x, o["counts"], o["seg_start"],
                   o["perm"], o["inv_perm"], o["n_res"], o["off_rows"], o["off_w"])
    y = torch.zeros((T * k + S * T, H), dtype=torch.float32, device="cuda")
    moe.moe_grouped_ffn(dev.dims, dev.x, o["perm"], o["counts"], o["seg_start"], dev.expert_slot, dev.w13, dev.w2,
                        dev.ws13, dev.ws2, y, dev.ws)
    out = torch.empty((T, H), dtype=o["out"].dtype, device="cuda")
    moe.moe_combine(dev.dims, o["topk_idx"], o["topk_w"], o["inv_perm"], dev.expert_slot, y,
                    y_off, o["n_res"], out, o["out_dtype"])
    return o, y, out


@pytest.mark.parametrize("name", ["c2_mixtral_decode", "c3_shared_decode", "c4_prefill", "c1_tiny_f32"])
def test_determinism_and_standalone_chain(moe, name):
    """Two fused runs are bitwise identical, and equal to the four-call chain bit for bit."""
    from paper_2608_21614_amd.device import DeviceLayer
    say("determinism + chain", name)
    dev = DeviceLayer(SyntheticLayer(CONFIGS[name], 3))
    o1 = dev.alloc_outputs()
    o2 = dev.alloc_outputs()
    dev.forward(o1)
    dev.forward(o2)
    _, _, out3 = _standalone_chain(moe, dev)
    torch.cuda.synchronize()
    a, b, c = _host(o1["out"]), _host(o2["out"]), _host(out3)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(a, c)


def test_host_merge_full_output_c3(moe):
    """Offloaded rows computed by the oracle (the host's role) merged by moe_combine: full layer output."""
    from paper_2608_21614_amd.device import DeviceLayer
    say("host merge c3 seed 4")
    lay = SyntheticLayer(CONFIGS["c3_shared_decode"], 4)
    dev = DeviceLayer(lay)
    o, y, _ = _standalone_chain(moe, dev)
    torch.cuda.synchronize()
    c = lay.cfg
    lg_ref = oracle.router_logits(lay.x, lay.w_router, lay.bias)
    idx = _host(o["topk_idx"])
    exp_idx, _ = expected_routing(lg_ref, idx, c.top_k)
    np.testing.assert_array_equal(idx, exp_idx)
    ref = oracle.layer_forward_synthetic(lay, idx=exp_idx)
    n_res = int(_host(o["n_res"])[0])
    P = c.tokens * c.top_k
    assert n_res == ref["n_res"] and n_res < P
    # grouped FFN rows vs the oracle's per-row expert outputs
    yr = _host(y)
    assert rel_l2(yr[:n_res], ref["y_rows"][:n_res]) <= TOL["bf16"]
    y_off = _dev(ref["y_rows"][n_res:P].astype(np.float32))
    out = torch.empty((c.tokens, c.hidden), dtype=torch.float32, device="cuda")
    moe.moe_combine(dev.dims, o["topk_idx"], o["topk_w"], o["inv_perm"], dev.expert_slot, y, y_off, o["n_res"], out,
                    moe.MOE_F32)
    torch.cuda.synchronize()
    full = ref["out_res"] + ref["out_off"]
    err = rel_l2(host_f64(out), full)
    say(f"  full-output rel-L2 {err:.3e}")
    assert err <= TOL["bf16"]


def test_stage_accumulate(moe):
    say("stage accumulate")
    counts = _dev(np.array([3, 0, 5, 1], np.int32))
    log = _dev(np.array([10, 20, 30, 2**40], np.int64))
    moe.moe_stage_accumulate(4, counts, log)
    moe.moe_stage_accumulate(4, counts, log)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(_host(log), [16, 20, 40, 2**40 + 2])


def test_read_probe_runs_and_keeps_sink(moe):
    """The streaming-read probe (a measurement utility) reads a buffer once and leaves the sink alone."""
    say("read probe")
    src = torch.zeros(1 << 22, dtype=torch.float32, device="cuda")      # 16 MiB of zeros: the xor is 0
    sink = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    moe.moe_read_probe(src, sink)
    moe.moe_read_probe(src, sink, nbytes=16 * 1001)                       # a ragged tail of chunks
    moe.moe_read_probe(src, sink, nbytes=0)
    torch.cuda.synchronize()
    assert int(sink.item()) == 7
