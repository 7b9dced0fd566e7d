"""Stage-boundary detection (Section IV-B.1): the cue machine against the oracle (CPU only).

The oracle (``oracle.cue_matches``) is the definition -- every cue compared with
the tail of every window -- and is pinned here on hand-worked streams and on a
library routine (numpy's sliding windows) for single cues.  The library's
automaton (``moe_cue_build`` / ``moe_cue_step``), fed one token per sequence
per step, must then report exactly the oracle's match at every step.
"""
import numpy as np
import pytest

import oracle
import workloads


def _lib():
    import paper_2608_21614_amd as saem
    return saem


def _run_machine(cues, stream):
    saem = _lib()
    fsm = saem.moe_cue_build(cues)
    s = np.asarray(stream, dtype=np.int32)
    if s.ndim == 1:
        s = s[:, None]
    state = np.zeros(s.shape[1], dtype=np.int32)
    out = np.empty_like(s)
    for i in range(s.shape[0]):
        out[i] = saem.moe_cue_step(fsm, s[i], state)
    return out


# ---------------------------------------------------------------- oracle pins

def test_oracle_hand_worked_stream():
    # cue ids: 0 = [5], 1 = [2, 3], 2 = [1, 2, 3]; the longest cue wins, not the lowest id
    got = oracle.cue_matches([[5], [2, 3], [1, 2, 3]], np.array([1, 2, 3, 4, 5, 2, 3, 3])).ravel()
    assert got.tolist() == [-1, -1, 2, -1, 0, -1, 1, -1]


def test_oracle_partial_match_falls_back_to_a_shorter_cue():
    # [1, 2, 3, 4] breaks at 5; the tail [2, 3, 5] is still a cue
    got = oracle.cue_matches([[1, 2, 3, 4], [2, 3, 5]], np.array([1, 2, 3, 5, 1, 2, 3, 4])).ravel()
    assert got.tolist() == [-1, -1, -1, 1, -1, -1, -1, 0]


def test_oracle_order_overlap_restart_and_duplicates():
    # token order matters: [1, 2] does not match 2, 1
    assert oracle.cue_matches([[1, 2]], np.array([2, 1, 2])).ravel().tolist() == [-1, -1, 0]
    # overlapping occurrences all count
    assert oracle.cue_matches([[7, 7]], np.array([7, 7, 7])).ravel().tolist() == [-1, 0, 0]
    # a negative token restarts the window: no match may span it
    assert oracle.cue_matches([[1, 2, 3]], np.array([1, 2, -1, 3, 1, 2, 3])).ravel().tolist() == \
        [-1, -1, -1, -1, -1, -1, 0]
    # identical cues report the lowest id
    assert oracle.cue_matches([[4, 4], [9], [4, 4]], np.array([4, 4])).ravel().tolist() == [-1, 0]
    # sequences are independent
    got = oracle.cue_matches([[1, 2]], np.array([[1, 2], [2, 1], [3, 2]]))
    assert got.tolist() == [[-1, -1], [0, -1], [-1, 0]]


def test_oracle_single_cue_equals_sliding_window_search():
    rng = np.random.default_rng(3)
    stream = rng.integers(0, 3, size=400)
    for cue in ([0], [1, 2], [2, 2, 1], [0, 1, 0, 1]):
        L = len(cue)
        win = np.lib.stride_tricks.sliding_window_view(stream, L)
        want = np.full(stream.size, -1)
        want[L - 1:][np.all(win == np.asarray(cue), axis=1)] = 0
        assert np.array_equal(oracle.cue_matches([cue], stream).ravel(), want)


def test_oracle_stage_lengths_from_events():
    m = np.full((10, 3), -1)
    m[2, 1] = 0       # stage ends after step 2
    m[2, 0] = 4       # same step in another sequence: one event
    m[6, 2] = 1
    m[9, 0] = 3       # last step: no new stage
    assert oracle.stage_lengths_from_events(m, 10).tolist() == [3, 4, 3]
    assert oracle.stage_lengths_from_events(np.full((5, 2), -1), 5).tolist() == [5]


# ---------------------------------------------------------------- library vs oracle

@pytest.mark.parametrize("seed", range(8))
def test_machine_matches_oracle_on_random_cues(seed):
    rng = np.random.default_rng(100 + seed)
    V = int(rng.integers(2, 6))                  # tiny vocabulary: many partial and full matches
    cues = []
    for _ in range(int(rng.integers(1, 9))):
        cues.append(rng.integers(0, V, size=int(rng.integers(1, 6))).tolist())
    if seed % 2 == 0 and len(cues) > 1:          # prefixes, suffixes and duplicates of other cues
        cues.append(cues[0][:max(1, len(cues[0]) - 1)])
        cues.append(cues[-2][1:] or cues[-2])
        cues.append(list(cues[0]))
    B = int(rng.integers(1, 9))
    stream = rng.integers(0, V, size=(300, B))
    stream[rng.random(stream.shape) < 0.02] = -1   # idle steps restart a window
    assert np.array_equal(_run_machine(cues, stream), oracle.cue_matches(cues, stream))


def test_machine_on_the_trace_stream_finds_every_planted_boundary():
    tr = workloads.StageTrace(workloads.TRACE, 0)
    ts = tr.token_stream()
    got = _run_machine(ts["cues"], ts["stream"])
    want = oracle.cue_matches(ts["cues"], ts["stream"])
    assert np.array_equal(got, want)
    events = set(np.flatnonzero((got >= 0).any(axis=1)).tolist())
    assert set(ts["planted"].tolist()) <= events
    # every planted cue ends a stage of the trace
    assert np.array_equal(ts["planted"], tr.stage_ends()[:-1])


def test_machine_without_cues_never_matches():
    saem = _lib()
    fsm = saem.moe_cue_build([])
    state = np.zeros(4, dtype=np.int32)
    for t in range(5):
        assert (saem.moe_cue_step(fsm, np.full(4, t, dtype=np.int32), state) == -1).all()


def test_machine_rejects_bad_input():
    saem = _lib()
    lib = saem.lib
    assert lib.moe_cue_fsm_words(-1) == -1
    assert lib.moe_cue_fsm_words(3) == 5 * 3 + 8
    buf = np.zeros(64, dtype=np.int32)
    off = np.array([0, 2, 2], dtype=np.int32)        # empty second cue
    tok = np.array([1, 2], dtype=np.int32)
    assert lib.moe_cue_build(2, off.ctypes.data, tok.ctypes.data, buf.ctypes.data, 64) == saem.MOE_ERR_INVALID_ARG
    off = np.array([0, 2], dtype=np.int32)
    tok = np.array([1, -3], dtype=np.int32)          # negative token id
    assert lib.moe_cue_build(1, off.ctypes.data, tok.ctypes.data, buf.ctypes.data, 64) == saem.MOE_ERR_INVALID_ARG
    off = np.array([1, 2], dtype=np.int32)           # offsets must start at 0
    assert lib.moe_cue_build(1, off.ctypes.data, tok.ctypes.data, buf.ctypes.data, 64) == saem.MOE_ERR_INVALID_ARG
    tok = np.array([1, 3], dtype=np.int32)
    off = np.array([0, 2], dtype=np.int32)
    small = np.zeros(17, dtype=np.int32)             # needs 5 * 2 + 8 = 18 words
    assert lib.moe_cue_build(1, off.ctypes.data, tok.ctypes.data, small.ctypes.data, 17) == saem.MOE_ERR_WORKSPACE
    assert not small.any()
    fsm = saem.moe_cue_build([[1, 3]])
    with pytest.raises(saem.MoeError):               # state out of range
        saem.moe_cue_step(fsm, np.array([1], dtype=np.int32), np.array([99], dtype=np.int32))
    junk = np.zeros_like(fsm)
    with pytest.raises(saem.MoeError):               # not a machine
        saem.moe_cue_step(junk, np.array([1], dtype=np.int32), np.zeros(1, dtype=np.int32))
    st = np.zeros(1, dtype=np.int32)
    m = np.zeros(1, dtype=np.int32)
    assert lib.moe_cue_step(fsm.ctypes.data, 1, None, st.ctypes.data, m.ctypes.data) == saem.MOE_ERR_INVALID_ARG
    assert lib.moe_cue_step(fsm.ctypes.data, 0, None, None, None) == saem.MOE_OK


@pytest.mark.parametrize("batch,mean", [(16, 2.0), (1, 1.5)])
def test_planted_cues_survive_short_stages(batch, mean):
    """Cues planted at boundaries a step or two apart never overwrite one another."""
    from dataclasses import replace
    cfg = replace(workloads.TRACE, steps=300, batch=batch, mean_stage_len=mean)
    for seed in range(6):
        ts = workloads.StageTrace(cfg, seed).token_stream()
        got = _run_machine(ts["cues"], ts["stream"])
        assert np.array_equal(got, oracle.cue_matches(ts["cues"], ts["stream"]))
        events = set(np.flatnonzero((got >= 0).any(axis=1)).tolist())
        assert set(ts["planted"].tolist()) <= events, seed
