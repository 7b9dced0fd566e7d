"""TC_seq, the paper's stage-to-stage routing coherence (Section III, Motivation 2), on the CPU.

The oracle writes the equation out; it is pinned on hand-worked traces and on
scipy's cosine distance.  The runtime's vectorised version (reported by the
trace bench) must equal it on random traces.
"""
import math

import numpy as np
import pytest
from scipy.spatial.distance import cosine

import oracle
from paper_2608_21614_amd.stage_trace import temporal_coherence


def test_oracle_hand_worked():
    # one layer, two experts: stage 1 routes only to expert 0, stage 2 evenly -> cos = 1/sqrt(2)
    counts = np.array([[[2, 0]], [[2, 0]], [[1, 1]]])
    assert math.isclose(oracle.temporal_coherence(counts, [2, 1]), 1 / math.sqrt(2), rel_tol=1e-15)
    # identical stages -> 1; disjoint experts -> 0
    assert math.isclose(oracle.temporal_coherence(np.array([[[3, 1]], [[6, 2]]]), [1, 1]), 1.0, rel_tol=1e-15)
    assert oracle.temporal_coherence(np.array([[[3, 0]], [[0, 5]]]), [1, 1]) == 0.0
    # two layers average; three stages average over the two transitions
    counts = np.array([[[1, 0], [1, 0]], [[1, 0], [0, 1]], [[0, 1], [0, 1]]])
    # transition 1: layer 0 cos 1, layer 1 cos 0 -> 0.5; transition 2: layer 0 cos 0, layer 1 cos 1 -> 0.5
    assert math.isclose(oracle.temporal_coherence(counts, [1, 1, 1]), 0.5, rel_tol=1e-15)
    assert math.isnan(oracle.temporal_coherence(counts, [3]))


def test_oracle_matches_scipy_cosine():
    rng = np.random.default_rng(7)
    counts = rng.integers(0, 9, size=(40, 3, 8))
    counts[:, :, 0] += 1                                   # no empty stage rows
    stage_len = [7, 13, 5, 15]
    ends = np.cumsum(stage_len)
    R = [counts[e - n:e].sum(axis=0) for e, n in zip(ends, stage_len)]
    want = np.mean([np.mean([1 - cosine(R[p][l], R[p + 1][l]) for l in range(3)]) for p in range(3)])
    assert math.isclose(oracle.temporal_coherence(counts, stage_len), want, rel_tol=1e-12)


@pytest.mark.parametrize("seed", range(5))
def test_runtime_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    L, E = int(rng.integers(1, 5)), int(rng.integers(2, 12))
    lens = rng.integers(1, 20, size=int(rng.integers(2, 8)))
    counts = rng.integers(0, 6, size=(int(lens.sum()), L, E))
    counts[:, :, int(rng.integers(E))] += 1
    assert math.isclose(temporal_coherence(counts, lens), oracle.temporal_coherence(counts, lens), rel_tol=1e-12)


@pytest.mark.parametrize("seed", range(5))
def test_runtime_clairvoyant_chr_matches_oracle_replay(seed):
    from paper_2608_21614_amd.stage_trace import clairvoyant_chr
    rng = np.random.default_rng(50 + seed)
    L, E = int(rng.integers(1, 5)), int(rng.integers(2, 12))
    n_slots = int(rng.integers(1, E + 1))
    lens = rng.integers(1, 20, size=int(rng.integers(1, 8)))
    counts = rng.integers(0, 4, size=(int(lens.sum()), L, E))    # small counts: many ties
    init = np.full((L, E), -1, np.int32)
    for l in range(L):
        init[l, rng.choice(E, n_slots, replace=False)] = np.arange(n_slots)
    ref = oracle.stage_replay(counts, lens, init, n_slots)
    assert clairvoyant_chr(counts, lens, n_slots) == ref["chr_clairvoyant"]
