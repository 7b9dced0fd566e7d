"""Stage-aware residency with real slot copies (SAEM Section IV-C) on the GPU.

A small stage-structured trace (2 layers, 96 steps, short stages) runs through
``StageResidencyRunner``: every call's fused layer forward, the device activation
logs, the plan at each boundary, and the copies of incoming experts' weights into
their slots on a copy stream, overlapping the next stage's first ``lag`` steps.

Checked against the oracle (routing counts from the device, as in the full trace
test, since routing does not depend on residency):
* the residency map each call ran with == oracle.stage_replay(..., lag)'s;
* the resident pairs of every call and the online CHR;
* every slot's bytes == the packed weights of the expert the plan put there;
* the routing of sampled calls (near ties resolved to a valid alternative) and
  their layer output == the oracle's resident partial sum under that routing.

With ``detect``, the boundaries come from the cue machine fed the batch's
generated tokens after every step (Section IV-B.1), on a token stream with a
small vocabulary so that background text also completes cues: the runner's
boundaries must be the oracle's cue events, and the replay runs over the stages
those events delimit, not the trace's true ones.
"""
from __future__ import annotations

from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle
from gpu_support import TOL, expected_routing, host_f64, rel_l2
from workloads import TRACE, StageTrace

pytestmark = pytest.mark.gpu

SMALL = replace(TRACE, layers=2, steps=96, hidden=256, ffn=512, mean_stage_len=12.0)


def say(*a):
    print("[residency]", *a, flush=True)


@pytest.mark.parametrize("lag,detect", [(0, False), (3, False), (2, True)])
def test_stage_residency_with_slot_copies(lag, detect):
    import paper_2608_21614_amd as moe
    from paper_2608_21614_amd.device import to_device
    from paper_2608_21614_amd.residency import StageResidencyRunner
    c = replace(SMALL, vocab=200, cue_min_rank=10) if detect else SMALL
    trace = StageTrace(c, seed=1)
    L, E, T, k, H = c.layers, c.experts, c.batch, c.top_k, c.hidden
    layers = [trace.layer(l) for l in range(L)]
    say(f"lag {lag}: {c.steps} steps x {L} layers, {trace.n_stages} stages {trace.stage_len.tolist()}")
    ends = trace.stage_ends()
    sample = [(0, 0), (int(ends[0]) + 1, 1), (min(int(ends[1]) + 2, c.steps - 1), 0), (c.steps - 1, 1)]
    run = StageResidencyRunner(trace, [lay.w_router for lay in layers],
                               lambda l, e: (layers[l].w13(e), layers[l].w2(e)), trace.x, lag=lag)
    detector, stage_len = None, trace.stage_len
    if detect:
        ts = trace.token_stream()
        detector = {"cues": ts["cues"], "stream": ts["stream"]}
        matched = oracle.cue_matches(ts["cues"], ts["stream"])
        stage_len = oracle.stage_lengths_from_events(matched, c.steps)
        say(f"detected stages {stage_len.tolist()} (true {trace.stage_len.tolist()})")
        assert len(stage_len) > trace.n_stages            # false positives split true stages
    r = run.run(keep_outputs=sample, detector=detector)
    np.testing.assert_array_equal(r["boundary_steps"], np.cumsum(stage_len)[:-1] - 1)
    say(f"CHR {r['chr_online']:.4f}, {r['copied_experts']} experts copied at {r['boundaries_with_copies']} "
        f"boundaries, stall {r['stall_ms_total']:.3f} ms")
    assert r["copied_experts"] > 0

    init = np.full((L, E), -1, np.int32)
    for l in range(L):
        ids = np.flatnonzero(trace.initial_resident[l])
        init[l, ids] = np.arange(len(ids))
    ref = oracle.stage_replay(r["counts"], stage_len, init, c.n_slots, lag=lag)
    np.testing.assert_array_equal(r["slot_history"], ref["slot_history"])
    np.testing.assert_array_equal(r["used_slot"] >= 0, ref["resident"])
    np.testing.assert_array_equal(r["n_res"], (r["counts"] * ref["resident"]).sum(axis=2))
    assert r["chr_online"] == ref["chr_online"]

    # slot contents: the packed weights of the expert each slot holds at the end
    for l in range(L):
        for e in np.flatnonzero(run.slot[l] >= 0):
            s = int(run.slot[l, e])
            for got, host in ((run.w13[l][s], layers[l].w13(int(e))), (run.w2[l][s], layers[l].w2(int(e)))):
                want = torch.empty_like(got)
                moe.moe_pack_weights(to_device(host), want)
                assert torch.equal(got, want), (l, int(e), s)

    # sampled calls: routing (near ties resolved as elsewhere) and the resident partial output
    stage_of = trace.stage_of_step()
    for step, l in sample:
        s = int(stage_of[step])
        x = trace.x(step, l)
        bias = trace.stage_bias[s, l]
        lg = oracle.router_logits(x, layers[l].w_router, bias)
        idx_dev = r["topk_idx"][(step, l)]
        # the device's routing: the oracle's, or (near-tied tokens) one of the valid alternatives
        idx, alts = expected_routing(lg, idx_dev, k)
        np.testing.assert_array_equal(idx_dev, idx)
        np.testing.assert_array_equal(np.bincount(idx.ravel(), minlength=E), r["counts"][step, l])
        resident = r["used_slot"][step, l] >= 0
        ref_out = oracle.layer_forward(x, layers[l].w_router, bias, resident, k, layers[l].w13, layers[l].w2,
                                       idx=idx, offloaded=False)
        err = rel_l2(host_f64(r["outputs"][(step, l)]), ref_out["out_res"])
        say(f"  step {step} layer {l}: resident {np.flatnonzero(resident).tolist()}, rel-L2 {err:.3e}")
        assert err <= TOL["bf16"]
