"""Pins of the CPU oracle to facts outside itself (no GPU).

Each test checks the oracle against something the paper or the mathematics
fixes: the paper's worked repacking example, closed forms, special cases that
reduce to a library routine, invariants, and brute force on tiny inputs.  The
set is chosen so that a dropped term, a wrong sign or index, or a transposed
operand anywhere in the oracle fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from workloads import bf16_bits_to_f32, f32_to_bf16_bits, make_layer

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------
# routing: router scores
# ----------------------------------------------------------------------------

def test_router_one_hot_reads_weight_rows_and_bias():
    """A one-hot token x = e_h scores expert e with w_router[e, h] + b[e] (catches a transposed router)."""
    H, E = 6, 4
    w = (np.arange(E * H, dtype=np.float32).reshape(E, H) - 7.0) / 4.0
    b = np.array([0.5, -1.0, 0.25, 2.0], dtype=np.float32)
    x = np.eye(H, dtype=np.float32)
    lg = oracle.router_logits(x, w, b)
    assert lg.shape == (H, E)
    np.testing.assert_array_equal(lg, w.T.astype(np.float64) + b.astype(np.float64))
    lg0 = oracle.router_logits(x, w, None)
    np.testing.assert_array_equal(lg0, w.T.astype(np.float64))


def test_router_bf16_inputs_are_read_exactly():
    """bf16 bit patterns 0x3F80=1, 0xC000=-2, 0x3E00=0.125, 0x4040=3 give an exactly known score."""
    x = np.array([[0x3F80, 0xC000, 0x3E00, 0x4040]], dtype=np.uint16)  # 1, -2, 0.125, 3
    w = np.array([[0x4040, 0x3F80, 0xC000, 0x3E00],                     # 3, 1, -2, 0.125
                  [0x3F80, 0x3F80, 0x3F80, 0x3F80]], dtype=np.uint16)
    lg = oracle.router_logits(x, w, np.array([0.0, 1.0], dtype=np.float32))
    assert lg[0, 0] == 1 * 3 + (-2) * 1 + 0.125 * (-2) + 3 * 0.125  # 1.125
    assert lg[0, 1] == 1 - 2 + 0.125 + 3 + 1.0


def test_router_matches_fp64_matmul_on_random_bf16():
    lay = make_layer(tokens=5, hidden=64, experts=7, ffn=64, top_k=2, dtype="bf16", seed=3)
    lg = oracle.router_logits(lay.x, lay.w_router, None)
    ref = bf16_bits_to_f32(lay.x).astype(np.float64) @ bf16_bits_to_f32(lay.w_router).astype(np.float64).T
    np.testing.assert_allclose(lg, ref, rtol=1e-13, atol=1e-13)


# ----------------------------------------------------------------------------
# routing: top-k and gate
# ----------------------------------------------------------------------------

def test_topk_closed_form_tie_to_lower_index():
    """Scores [1,3,2,3], k=2: the two 3s tie; order is expert 1 then 3; weights 1/2 each."""
    idx, w = oracle.topk(np.array([[1.0, 3.0, 2.0, 3.0]]), 2)
    assert idx.tolist() == [[1, 3]]
    assert w.tolist() == [[0.5, 0.5]]


def test_topk_closed_form_weights():
    """Scores [0, ln 3, -inf, -1], k=2: experts 1 then 0 with weights 3/4 and 1/4."""
    idx, w = oracle.topk(np.array([[0.0, math.log(3.0), -math.inf, -1.0]]), 2)
    assert idx.tolist() == [[1, 0]]
    np.testing.assert_allclose(w, [[0.75, 0.25]], rtol=1e-15)


def test_topk_all_equal_and_all_minus_inf():
    for val in (0.0, 2.5, -math.inf):
        idx, w = oracle.topk(np.full((3, 6), val), 4)
        assert idx.tolist() == [[0, 1, 2, 3]] * 3
        np.testing.assert_array_equal(w, np.full((3, 4), 0.25))


def test_topk_k1_is_argmax_with_weight_one():
    rng = np.random.default_rng(0)
    lg = rng.standard_normal((50, 9))
    lg[3, [2, 5]] = 10.0  # a tie at the top: np.argmax takes the first
    idx, w = oracle.topk(lg, 1)
    np.testing.assert_array_equal(idx[:, 0], np.argmax(lg, axis=1))
    np.testing.assert_array_equal(w, np.ones((50, 1)))


def test_topk_k_equals_E_is_full_softmax():
    rng = np.random.default_rng(1)
    lg = rng.standard_normal((20, 8)) * 3
    idx, w = oracle.topk(lg, 8)
    np.testing.assert_array_equal(idx, np.argsort(-lg, axis=1, kind="stable"))
    sm = scipy.special.softmax(lg, axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(sm, idx.astype(np.int64), axis=1), rtol=1e-13)


def test_topk_matches_stable_argsort_and_renormalised_softmax():
    rng = np.random.default_rng(2)
    lg = np.round(rng.standard_normal((200, 16)), 1)  # coarse values: many ties
    for k in (1, 2, 3, 6, 16):
        idx, w = oracle.topk(lg, k)
        np.testing.assert_array_equal(idx, np.argsort(-lg, axis=1, kind="stable")[:, :k])
        sel = np.take_along_axis(lg, idx.astype(np.int64), axis=1)
        np.testing.assert_allclose(w, scipy.special.softmax(sel, axis=1), rtol=1e-13)
        np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=1e-14)
        # gate over the top-k equals the full softmax renormalised over the selection
        full = np.take_along_axis(scipy.special.softmax(lg, axis=1), idx.astype(np.int64), axis=1)
        np.testing.assert_allclose(w, full / full.sum(axis=1, keepdims=True), rtol=1e-12)


def test_topk_invariant_to_constant_shift():
    rng = np.random.default_rng(3)
    lg = rng.standard_normal((40, 10))
    i0, w0 = oracle.topk(lg, 3)
    i1, w1 = oracle.topk(lg + 7.0, 3)
    np.testing.assert_array_equal(i0, i1)
    np.testing.assert_allclose(w0, w1, rtol=1e-12)


# ----------------------------------------------------------------------------
# repacking
# ----------------------------------------------------------------------------

def _logits_for_routing(routing, E):
    """Scores under which each token's listed experts are its top-k, in the listed order."""
    T = len(routing)
    lg = np.zeros((T, E))
    for t, es in enumerate(routing):
        for r, e in enumerate(es):
            lg[t, e] = 10.0 - r
    return lg


def test_repack_paper_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "repack_worked_example.json")))
    idx, _ = oracle.topk(_logits_for_routing(g["routing"], g["experts"]), g["top_k"])
    assert idx.tolist() == g["routing"]
    rp = oracle.repack(idx, np.ones(g["experts"], dtype=bool))
    k = g["top_k"]
    for e, toks in g["expected_tokens_per_expert"].items():
        e = int(e)
        rows = rp["perm"][rp["seg_start"][e]: rp["seg_start"][e] + rp["counts"][e]]
        assert (rows // k).tolist() == toks
    d = g["derived_under_canonical_order"]
    assert rp["counts"].tolist() == d["counts"]
    assert rp["seg_start"].tolist() == d["seg_start"]
    assert (rp["perm"] // k).tolist() == d["perm_token"]
    assert rp["n_res"] == 8


def test_repack_worked_example_with_offloaded_experts():
    """E1 and E3 offloaded: resident groups E0, E2 first, then E1, E3."""
    g = json.load(open(os.path.join(GOLDEN, "repack_worked_example.json")))
    idx = np.array(g["routing"], dtype=np.int32)
    rp = oracle.repack(idx, np.array([1, 0, 1, 0], dtype=bool))
    assert rp["counts"].tolist() == [2, 2, 3, 1]
    assert rp["seg_start"].tolist() == [0, 5, 2, 7]
    assert (rp["perm"] // 2).tolist() == [0, 3, 0, 1, 3, 1, 2, 2]
    assert rp["n_res"] == 5


def _check_repack_against_library(idx, resident):
    T, k = idx.shape
    E = resident.size
    rp = oracle.repack(idx, resident)
    flat = idx.ravel().astype(np.int64)
    np.testing.assert_array_equal(rp["counts"], np.bincount(flat, minlength=E))
    q = np.arange(T * k)
    # stable sort of pairs by key (offloaded?, expert, pair index) -- a library routine
    ref_perm = np.lexsort((q, flat, ~resident[flat]))
    np.testing.assert_array_equal(rp["perm"], ref_perm)
    np.testing.assert_array_equal(rp["inv_perm"][rp["perm"]], q)
    assert rp["n_res"] == int(rp["counts"][resident].sum())
    for e in range(E):
        seg = rp["perm"][rp["seg_start"][e]: rp["seg_start"][e] + rp["counts"][e]]
        assert np.all(flat[seg] == e)
        assert np.all(np.diff(seg // k) > 0)
    assert np.all(resident[flat[rp["perm"][: rp["n_res"]]]])
    assert not np.any(resident[flat[rp["perm"][rp["n_res"]:]]])
    return rp


@pytest.mark.parametrize("T,E,k", [(1, 1, 1), (7, 8, 2), (64, 60, 4), (300, 64, 6), (33, 256, 8), (5, 3, 3)])
def test_repack_matches_lexsort_and_bincount(T, E, k):
    rng = np.random.default_rng(T * 1000 + E * 10 + k)
    idx = np.stack([rng.choice(E, k, replace=False) for _ in range(T)]).astype(np.int32)
    for resident in (np.ones(E, bool), np.zeros(E, bool), rng.random(E) < 0.5):
        _check_repack_against_library(idx, resident)


def test_repack_empty_batch_and_bad_index():
    rp = oracle.repack(np.zeros((0, 2), dtype=np.int32), np.ones(4, bool))
    assert rp["counts"].tolist() == [0, 0, 0, 0] and rp["n_res"] == 0 and rp["perm"].size == 0
    with pytest.raises(ValueError):
        oracle.repack(np.array([[0, 4]], dtype=np.int32), np.ones(4, bool))


# ----------------------------------------------------------------------------
# expert FFN
# ----------------------------------------------------------------------------

def _ffn_f32(x, w1, w3, w2):
    """Pack math-shaped W1 [H,F], W3 [H,F], W2 [F,H] into the stored layout and run the oracle."""
    x = np.asarray(x, np.float32)
    w13 = np.ascontiguousarray(np.concatenate([w1.T, w3.T], axis=0), dtype=np.float32)
    w2s = np.ascontiguousarray(w2.T, dtype=np.float32)
    return oracle.expert_ffn(x, np.arange(x.shape[0], dtype=np.int32), w13, w2s)


def test_ffn_scalar_closed_forms():
    """H = F = 1: y = c * silu(a v) * (b v), with silu(0)=0, silu(1)=e/(1+e), silu(+-ln 3)=+-(3/4, 1/4) ln 3."""
    cases = [
        (0.0, 1.0, 1.0, 1.0, 0.0),
        (1.0, 1.0, 1.0, 1.0, math.e / (1.0 + math.e)),
        (1.0, 1.0, -2.0, 0.5, -math.e / (1.0 + math.e)),
        (float(np.float32(math.log(3.0))), 1.0, 1.0, 1.0, 0.75 * math.log(3.0) * math.log(3.0)),
        (float(np.float32(math.log(3.0))), -1.0, 1.0, 1.0, -0.25 * math.log(3.0) * math.log(3.0)),
    ]
    for v, a, b, c, want in cases:
        y = _ffn_f32([[v]], np.array([[a]]), np.array([[b]]), np.array([[c]]))
        assert y.shape == (1, 1)
        np.testing.assert_allclose(y[0, 0], want, rtol=2e-7, atol=1e-15)


def test_ffn_permutation_weights_closed_form():
    """W1 = 2*P_a, W3 = diag(d), W2 = P_b for permutation matrices: y follows the index maps.

    (x W1)[f] = 2 x[pa^-1(f)] where P_a[h, pa(h)] = 1; a transposed operand permutes the wrong way.
    """
    H = F = 5
    pa = np.array([2, 0, 4, 1, 3])
    pb = np.array([1, 3, 0, 4, 2])
    Pa = np.zeros((H, F)); Pa[np.arange(H), pa] = 1
    Pb = np.zeros((F, H)); Pb[np.arange(F), pb] = 1
    d = np.array([1.0, -2.0, 0.5, 3.0, -1.0])
    x = np.array([[0.5, -1.0, 2.0, 0.0, 1.5]])
    y = _ffn_f32(x, 2 * Pa, np.diag(d), Pb)
    inv_pa = np.argsort(pa)
    a = np.empty(F)
    for f in range(F):
        g = 2 * x[0, inv_pa[f]]
        a[f] = g / (1 + math.exp(-g)) * (x[0, f] * d[f])
    want = np.empty(H)
    for f in range(F):
        want[pb[f]] = a[f]
    np.testing.assert_allclose(y[0], want, rtol=1e-12, atol=1e-15)


def _random_expert(H, F, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((4, H)).astype(np.float32), rng.standard_normal((H, F)).astype(np.float32) * 0.3,
            rng.standard_normal((H, F)).astype(np.float32) * 0.3, rng.standard_normal((F, H)).astype(np.float32) * 0.3)


def test_ffn_gate_sign_identity():
    """silu(z) - silu(-z) = z gives y(-W1) - y(W1) = -((x W1) * (x W3)) W2.

    Pins which projection is gated and the sign of both: swapping W1 and W3
    makes y(-W1) = -y(W1) instead.
    """
    x, w1, w3, w2 = _random_expert(6, 10, 4)
    y = _ffn_f32(x, w1, w3, w2)
    ym = _ffn_f32(x, -w1, w3, w2)
    X = x.astype(np.float64)
    rhs = -((X @ w1.astype(np.float64)) * (X @ w3.astype(np.float64))) @ w2.astype(np.float64)
    np.testing.assert_allclose(ym - y, rhs, rtol=1e-10, atol=1e-12)


def test_ffn_linear_in_up_and_down_projections():
    x, w1, w3, w2 = _random_expert(8, 12, 5)
    y = _ffn_f32(x, w1, w3, w2)
    np.testing.assert_allclose(_ffn_f32(x, w1, 2 * w3, w2), 2 * y, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(_ffn_f32(x, w1, w3, -0.5 * w2), -0.5 * y, rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(_ffn_f32(x, np.zeros_like(w1), w3, w2), np.zeros_like(y))


def test_ffn_matches_torch_silu_mlp_fp64():
    x, w1, w3, w2 = _random_expert(16, 24, 6)
    y = _ffn_f32(x, w1, w3, w2)
    X, W1, W3, W2 = (torch.from_numpy(a.astype(np.float64)) for a in (x, w1, w3, w2))
    ref = (torch.nn.functional.silu(X @ W1) * (X @ W3)) @ W2
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-12, atol=1e-13)


def test_ffn_row_token_gathers_rows():
    x, w1, w3, w2 = _random_expert(8, 8, 7)
    w13 = np.ascontiguousarray(np.concatenate([w1.T, w3.T]), dtype=np.float32)
    w2s = np.ascontiguousarray(w2.T)
    full = oracle.expert_ffn(x, np.arange(4, dtype=np.int32), w13, w2s)
    sub = oracle.expert_ffn(x, np.array([3, 1, 3], dtype=np.int32), w13, w2s)
    np.testing.assert_array_equal(sub, full[[3, 1, 3]])


# ----------------------------------------------------------------------------
# whole layer
# ----------------------------------------------------------------------------

def _dense_moe_reference(lay):
    """Dense form of the MoE layer: every expert on every token, weighted by a sparse gate matrix.

    Gate matrix from a stable argsort (selection) and scipy's softmax (weights);
    expert MLPs with torch fp64 silu and matmul.  No repacking, no residency.
    """
    c = lay.cfg
    cvt = (lambda a: bf16_bits_to_f32(a)) if c.dtype == "bf16" else (lambda a: a)
    X = torch.from_numpy(cvt(lay.x).astype(np.float64))
    lg = X.numpy() @ cvt(lay.w_router).astype(np.float64).T
    if lay.bias is not None:
        lg = lg + lay.bias.astype(np.float64)
    sel = np.argsort(-lg, axis=1, kind="stable")[:, : c.top_k]
    G = np.zeros_like(lg)
    np.put_along_axis(G, sel, scipy.special.softmax(np.take_along_axis(lg, sel, axis=1), axis=1), axis=1)
    out = torch.zeros_like(X)
    for e in range(c.experts):
        w13 = torch.from_numpy(cvt(lay.w13(e)).astype(np.float64))
        w2 = torch.from_numpy(cvt(lay.w2(e)).astype(np.float64))
        F = c.ffn
        y = (torch.nn.functional.silu(X @ w13[:F].T) * (X @ w13[F:].T)) @ w2.T
        out += torch.from_numpy(G[:, e:e + 1]) * y
    for s in range(c.shared):
        w13 = torch.from_numpy(cvt(lay.ws13(s)).astype(np.float64))
        w2 = torch.from_numpy(cvt(lay.ws2(s)).astype(np.float64))
        Fs = c.shared_ffn
        out += (torch.nn.functional.silu(X @ w13[:Fs].T) * (X @ w13[Fs:].T)) @ w2.T
    return lg, sel, out.numpy()


@pytest.mark.parametrize("dtype,shared,resident", [("f32", 0, 8), ("bf16", 0, 3), ("bf16", 2, 5), ("f32", 1, 0)])
def test_layer_matches_dense_moe_brute_force(dtype, shared, resident):
    lay = make_layer(tokens=9, hidden=32, experts=8, ffn=48, top_k=3, dtype=dtype, shared=shared,
                     shared_ffn=40, n_resident=resident, residency="random", seed=11)
    lg, sel, dense = _dense_moe_reference(lay)
    o = oracle.layer_forward_synthetic(lay)
    np.testing.assert_allclose(o["logits"], lg, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(o["idx"], sel)
    np.testing.assert_allclose(o["out_res"] + o["out_off"], dense, rtol=1e-10, atol=1e-12)
    if resident == 8:
        assert not o["out_off"].any()
    if resident == 0 and shared == 0:
        assert not o["out_res"].any()


def test_layer_single_expert_k1_is_dense_mlp():
    lay = make_layer(tokens=6, hidden=16, experts=1, ffn=20, top_k=1, dtype="f32", seed=12)
    o = oracle.layer_forward_synthetic(lay)
    assert (o["idx"] == 0).all() and (o["w"] == 1).all()
    X = torch.from_numpy(lay.x.astype(np.float64))
    w13 = torch.from_numpy(lay.w13(0).astype(np.float64))
    ref = (torch.nn.functional.silu(X @ w13[:20].T) * (X @ w13[20:].T)) @ torch.from_numpy(lay.w2(0).astype(np.float64)).T
    np.testing.assert_allclose(o["out_res"], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_layer_shared_experts_added_with_unit_weight():
    """Routed down projections zeroed: the output is exactly the sum of the shared experts."""
    lay = make_layer(tokens=5, hidden=16, experts=4, ffn=8, top_k=2, dtype="f32", shared=2, shared_ffn=12, seed=13)
    zero = np.zeros((16, 8), dtype=np.float32)
    o = oracle.layer_forward(lay.x, lay.w_router, None, lay.resident, 2, lay.w13, lambda e: zero,
                             2, lay.ws13, lay.ws2)
    want = sum(oracle.expert_ffn(lay.x, np.arange(5, dtype=np.int32), lay.ws13(s), lay.ws2(s)) for s in range(2))
    np.testing.assert_allclose(o["out_res"], want, rtol=1e-14)


def test_layer_sampled_tokens_match_full_batch():
    lay = make_layer(tokens=12, hidden=16, experts=6, ffn=8, top_k=2, dtype="bf16", shared=1, shared_ffn=8,
                     n_resident=3, residency="random", seed=14)
    full = oracle.layer_forward_synthetic(lay)
    samp = oracle.layer_forward_synthetic(lay, sample=[11, 0, 5])
    np.testing.assert_array_equal(samp["out_res"], full["out_res"][[11, 0, 5]])
    np.testing.assert_array_equal(samp["out_off"], full["out_off"][[11, 0, 5]])


def test_layer_independent_of_thread_count():
    """The oracle's loops split outputs, never sums: one thread gives the same bits."""
    lay = make_layer(24, 128, 8, 128, 2, dtype="bf16", shared=1, shared_ffn=64, n_resident=5, residency="random",
                     seed=4)
    n = oracle.threads()
    try:
        a = oracle.layer_forward_synthetic(lay, offloaded=True)
        oracle.set_threads(1)
        assert oracle.threads() == 1
        b = oracle.layer_forward_synthetic(lay, offloaded=True)
    finally:
        oracle.set_threads(n)
    for key in ("out_res", "out_off", "perm", "counts"):
        np.testing.assert_array_equal(a[key], b[key])


def test_layer_given_logits_and_selection():
    lay = make_layer(tokens=4, hidden=8, experts=4, ffn=8, top_k=2, dtype="f32", seed=15)
    g = json.load(open(os.path.join(GOLDEN, "repack_worked_example.json")))
    lg = _logits_for_routing(g["routing"], 4)
    o = oracle.layer_forward_synthetic(lay, logits=lg)
    assert o["idx"].tolist() == g["routing"]
    o2 = oracle.layer_forward_synthetic(lay, logits=lg, idx=np.array([[2, 0], [1, 2], [1, 3], [0, 2]]))
    assert o2["idx"].tolist()[0] == [2, 0]
    np.testing.assert_allclose(o2["w"][0], [math.exp(-1) / (1 + math.exp(-1)), 1 / (1 + math.exp(-1))])


def test_near_tie_alternatives():
    lg = np.array([[1.0, 3.0, 3.0 + 1e-7, 0.0], [5.0, 4.0, 3.0, 2.0], [1.0, 1.0, 1.0, 0.0]])
    alts = oracle.near_tie_alternatives(lg, 1, 1e-4)
    assert alts[0] == [(1,), (2,)]
    assert 1 not in alts
    assert alts[2] == [(0,), (1,), (2,)]
    alts2 = oracle.near_tie_alternatives(lg, 2, 1e-4)
    assert alts2[0] == [(1, 2), (2, 1)]


# ----------------------------------------------------------------------------
# stage-aware residency
# ----------------------------------------------------------------------------

def test_stage_plan_keeps_incumbent_slots():
    # top-2 = {1, 2}; incumbents 0 (slot 0) and 3 (slot 1) are evicted; 1 and 2 take slots 0, 1
    assert oracle.stage_plan(np.array([5, 9, 9, 1]), 2, np.array([0, -1, -1, 1])).tolist() == [-1, 0, 1, -1]
    # ties at 5: experts 0 and 1 win; 1 keeps slot 0, 0 takes the slot freed by 2
    assert oracle.stage_plan(np.array([5, 5, 5, 0]), 2, np.array([-1, 0, 1, -1])).tolist() == [1, 0, -1, -1]
    # unchanged set keeps its layout
    assert oracle.stage_plan(np.array([0, 7, 0, 3]), 2, np.array([-1, 1, -1, 0])).tolist() == [-1, 1, -1, 0]


def test_cache_hit_ratio_exact():
    counts = np.array([[3, 1, 0, 4], [0, 2, 2, 4]])
    res = np.array([[1, 0, 0, 1], [1, 1, 0, 0]], dtype=bool)
    assert oracle.cache_hit_ratio(counts, res) == (3 + 4 + 0 + 2) / 16


# ----------------------------------------------------------------------------
# generator
# ----------------------------------------------------------------------------

def test_bf16_rounding_round_to_nearest_even():
    """Halfway cases go to the even mantissa; agrees with torch's bf16 conversion."""
    vals = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -7 + 2 ** -9], dtype=np.float32)
    want = np.array([1.0, 1.0, 1.0 + 2 ** -6, -2.5, 1.0 + 2 ** -7], dtype=np.float32)
    got = bf16_bits_to_f32(f32_to_bf16_bits(vals))
    np.testing.assert_array_equal(got, want)
    rnd = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    np.testing.assert_array_equal(bf16_bits_to_f32(f32_to_bf16_bits(rnd)),
                                  torch.from_numpy(rnd).to(torch.bfloat16).float().numpy())


def test_generator_is_deterministic_and_thread_independent(monkeypatch):
    import workloads
    a = make_layer(tokens=3, hidden=64, experts=4, ffn=600, top_k=2, seed=21).w13(2)
    monkeypatch.setattr(workloads, "_THREADS", 1)
    monkeypatch.setattr(workloads, "_CHUNK", 1 << 12)
    b = make_layer(tokens=3, hidden=64, experts=4, ffn=600, top_k=2, seed=21).w13(2)
    monkeypatch.setattr(workloads, "_THREADS", 4)
    c = make_layer(tokens=3, hidden=64, experts=4, ffn=600, top_k=2, seed=21).w13(2)
    np.testing.assert_array_equal(b, c)  # same chunking, different thread counts
    assert a.shape == b.shape
    d = make_layer(tokens=3, hidden=64, experts=4, ffn=600, top_k=2, seed=22).w13(2)
    assert not np.array_equal(a, d)


def test_stage_replay_hand_trace():
    """Two stages whose activation sets swap: the online policy lags one stage (CHR 0), the clairvoyant one hits all."""
    c = np.zeros((4, 1, 4), int)
    c[0, 0] = c[1, 0] = [3, 1, 0, 0]
    c[2, 0] = c[3, 0] = [0, 0, 2, 2]
    r = oracle.stage_replay(c, np.array([2, 2]), np.array([[-1, -1, 0, 1]]), 2)
    assert r["slot_history"].tolist() == [[[-1, -1, 0, 1]], [[0, 1, -1, -1]]]
    assert r["chr_online"] == 0.0 and r["chr_clairvoyant"] == 1.0


def test_stage_replay_stable_routing_and_exact_ratio():
    """Routing fixed on experts {1, 3}: after the first stage the online policy is as good as the clairvoyant one."""
    c = np.zeros((6, 2, 4), int)
    c[:, :, 1] = 5
    c[:, :, 3] = 3
    r = oracle.stage_replay(c, np.array([1, 2, 3]), np.array([[0, 1, -1, -1], [0, 1, -1, -1]]), 2)
    # stage 0 (1 step): resident {0,1} -> hits 5 of 8 per call; stages 1-2: resident {1,3} -> 8 of 8
    assert r["chr_online"] == (2 * 5 + 10 * 8) / (12 * 8)
    assert r["chr_clairvoyant"] == 1.0
    assert r["resident"][1:].all(axis=0)[:, [1, 3]].all()


def test_stage_replay_prefetch_lag_hand_trace():
    """Copies overlapped with the next stage's first steps (Section IV-C.3): during the first
    `lag` steps of a stage only the experts that keep their slot are resident."""
    c = np.zeros((8, 1, 4), int)
    c[0:2, 0] = [3, 1, 0, 0]          # stage 0 (2 steps): log [6, 2, 0, 0] -> keep {0, 1}
    c[2:5, 0] = [0, 2, 2, 0]          # stage 1 (3 steps): log [0, 6, 6, 0] -> {1 stays, 2 enters slot 0}
    c[5:8, 0] = [0, 0, 1, 5]          # stage 2 (3 steps)
    init = np.array([[0, 1, -1, -1]])
    lens = np.array([2, 3, 3])
    r0 = oracle.stage_replay(c, lens, init, 2)
    assert r0["slot_history"][2].tolist() == [[-1, 1, 0, -1]]
    assert r0["chr_online"] == (8 + 6 + 3) / 38
    r2 = oracle.stage_replay(c, lens, init, 2, lag=2)
    assert r2["chr_online"] == (8 + 6 + 1) / 38
    assert r2["resident"][5, 0].tolist() == [False, True, False, False]
    assert r2["resident"][6, 0].tolist() == [False, True, False, False]
    assert r2["resident"][7, 0].tolist() == [False, True, True, False]
    # stage 1 keeps stage 0's map: the lag changes nothing there
    assert (r2["resident"][2:5] == r0["resident"][2:5]).all()
    # a lag longer than the stage: the incoming expert never serves a pair in it
    r9 = oracle.stage_replay(c, lens, init, 2, lag=9)
    assert r9["chr_online"] == (8 + 6 + 0) / 38
    assert r9["chr_clairvoyant"] == r0["chr_clairvoyant"]
