"""CPU oracle for one MoE layer's forward (SAEM, arXiv 2608.21614).

TEST INFRASTRUCTURE ONLY.  The test suite, the package smoke check and the
bench's CPU-baseline leg may import this package; nothing on the product path
may.  It shares no code with the HIP library: the heavy loops are plain C in
``moe_oracle.c`` (fp64), the composition is here, and the only thing both sides
have in common is the seeded input buffers from ``workloads``.

The layer, in the paper's order (Section IV-A overview; Section IV-D.2 hybrid
CPU-GPU pipeline; Section IV-E.1 expert-aligned token repacking):

1. router scores and top-k gating (Section II-A);
2. expert-aligned repacking of the (token, expert) pairs (Section IV-E.1);
3. partition by the residency map into GPU-bound and host-bound rows
   (Section IV-D.2);
4. each expert once over its dense buffer (Section IV-E.1);
5. merge of the expert outputs back to token order (Section IV-D.2); the
   always-on shared experts are added with weight 1.

Readings where the paper is silent (renormalised softmax gate, SwiGLU expert,
lowest-index tie-break, canonical repack order, shared experts) are stated on
the functions below.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Callable, Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_DEFAULT_LIB = os.path.join(_HERE, "libmoe_oracle.so")
# an alternative build of the oracle (e.g. one with a planted mistake, to check that the pins catch it)
_LIB_PATH = os.environ.get("MOE_ORACLE_LIB", _DEFAULT_LIB)
_lib = None

F32, BF16 = 0, 1


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (fp64, OpenMP, no fast-math)."""
    if force or not os.path.exists(_DEFAULT_LIB):
        tmp = _DEFAULT_LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _DEFAULT_LIB)
    return _DEFAULT_LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(_LIB_PATH)
        i64, vp, dp, ip = ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
        lib.oracle_router_logits.argtypes = [i64, i64, i64, ctypes.c_int, vp, vp, vp, dp]
        lib.oracle_router_logits.restype = None
        lib.oracle_topk.argtypes = [i64, i64, i64, dp, ip, dp]
        lib.oracle_topk.restype = None
        lib.oracle_repack.argtypes = [i64, i64, i64, ip, vp, ip, ip, ip, ip, ip]
        lib.oracle_repack.restype = ctypes.c_int
        lib.oracle_expert_ffn.argtypes = [i64, i64, i64, ctypes.c_int, vp, ip, vp, vp, dp]
        lib.oracle_expert_ffn.restype = None
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        lib.oracle_set_threads.argtypes = [ctypes.c_int]
        lib.oracle_set_threads.restype = None
        _lib = lib
    return _lib


def threads() -> int:
    """OpenMP threads the oracle's loops run on."""
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Threads for later calls (results do not depend on it: loops split outputs, not sums)."""
    _load().oracle_set_threads(int(n))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return F32
    raise TypeError(f"oracle takes float32 or bf16 (uint16 bits) tensors, got {a.dtype}")


def router_logits(x: np.ndarray, w_router: np.ndarray, bias: Optional[np.ndarray]) -> np.ndarray:
    """Router scores x . w_router[e] + bias[e] in fp64 (Section II-A).  x [T,H], w_router [E,H]."""
    x = np.ascontiguousarray(x)
    w_router = np.ascontiguousarray(w_router)
    T, H = x.shape
    E = w_router.shape[0]
    assert w_router.shape[1] == H and x.dtype == w_router.dtype
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    out = np.empty((T, E), dtype=np.float64)
    _load().oracle_router_logits(T, H, E, _dtype_code(x), _ptr(x), _ptr(w_router), _ptr(b), _ptr(out))
    return out


def topk(logits: np.ndarray, k: int):
    """Top-k gate on given scores (Section II-A).

    Returns (idx [T,k] int32, w [T,k] fp64).  idx is ordered by decreasing score,
    equal scores to the lower expert index; w is the softmax over the k selected
    scores.  Scores are compared exactly as given (fp32 scores compare as their
    exact fp64 values).
    """
    lg = np.ascontiguousarray(logits, dtype=np.float64)
    T, E = lg.shape
    assert 1 <= k <= E
    idx = np.empty((T, k), dtype=np.int32)
    w = np.empty((T, k), dtype=np.float64)
    _load().oracle_topk(T, E, k, _ptr(lg), _ptr(idx), _ptr(w))
    return idx, w


def repack(idx: np.ndarray, resident: np.ndarray) -> Dict[str, np.ndarray]:
    """Expert-aligned repacking with the residency split (Sections IV-E.1, IV-D.2).

    Canonical order of packed rows: resident experts by ascending id, then
    offloaded experts by ascending id; inside an expert, ascending token.
    """
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    T, k = idx.shape
    res = np.ascontiguousarray(resident, dtype=np.uint8)
    E = res.shape[0]
    counts = np.empty(E, dtype=np.int32)
    seg = np.empty(E, dtype=np.int32)
    perm = np.empty(T * k, dtype=np.int32)
    inv = np.empty(T * k, dtype=np.int32)
    n_res = np.zeros(1, dtype=np.int32)
    rc = _load().oracle_repack(T, E, k, _ptr(idx), _ptr(res), _ptr(counts), _ptr(seg), _ptr(perm),
                               _ptr(inv), _ptr(n_res))
    if rc != 0:
        raise ValueError("expert index out of range")
    return {"counts": counts, "seg_start": seg, "perm": perm, "inv_perm": inv, "n_res": int(n_res[0])}


def group_order(resident: np.ndarray) -> np.ndarray:
    """Experts in packed-row order: resident ascending, then offloaded ascending."""
    res = np.asarray(resident, dtype=bool)
    return np.concatenate([np.flatnonzero(res), np.flatnonzero(~res)]).astype(np.int32)


def expert_ffn(x: np.ndarray, row_token: np.ndarray, w13: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """One SwiGLU expert over a dense buffer of rows (Section IV-E.1).

    y[r] = (silu(x[t] W1) * (x[t] W3)) W2 with t = row_token[r]; storage as in
    the C ABI: w13 [2F,H] (gate rows then up rows), w2 [H,F].  fp64 result.
    """
    x = np.ascontiguousarray(x)
    w13 = np.ascontiguousarray(w13)
    w2 = np.ascontiguousarray(w2)
    rt = np.ascontiguousarray(row_token, dtype=np.int32)
    T, H = x.shape
    F = w13.shape[0] // 2
    assert w13.shape == (2 * F, H) and w2.shape == (H, F)
    assert x.dtype == w13.dtype == w2.dtype
    assert rt.size == 0 or (rt.min() >= 0 and rt.max() < T)
    y = np.empty((rt.size, H), dtype=np.float64)
    _load().oracle_expert_ffn(rt.size, H, F, _dtype_code(x), _ptr(x), _ptr(rt), _ptr(w13), _ptr(w2), _ptr(y))
    return y


def layer_forward(x: np.ndarray, w_router: np.ndarray, bias: Optional[np.ndarray], resident: np.ndarray,
                  k: int, w13_of: Callable[[int], np.ndarray], w2_of: Callable[[int], np.ndarray],
                  n_shared: int = 0, ws13_of: Optional[Callable[[int], np.ndarray]] = None,
                  ws2_of: Optional[Callable[[int], np.ndarray]] = None,
                  logits: Optional[np.ndarray] = None, idx: Optional[np.ndarray] = None,
                  sample: Optional[Sequence[int]] = None, offloaded: bool = True) -> Dict[str, np.ndarray]:
    """The whole layer, steps 1-5 in the paper's order.

    logits: route these scores instead of computing them (fp32 scores are taken
            as their exact values).
    idx:    use this expert selection (a routing the caller already fixed, e.g.
            one of several valid choices for a near-tied token); the gate weights
            are still the softmax of the scores over the selection.
    sample: compute outputs only for these tokens (routing and repacking always
            cover the whole batch).
    offloaded: False skips the offloaded experts (out_off stays zero).

    Returns logits, idx, w, counts, seg_start, perm, inv_perm, n_res, and for the
    sampled tokens: out_res (resident routed experts + shared experts),
    out_off (offloaded routed experts), y_rows (each packed row's unweighted
    expert output, NaN for rows outside the sample).
    """
    T, H = x.shape
    E = w_router.shape[0]
    if logits is None:
        logits = router_logits(x, w_router, bias)
    logits = np.asarray(logits, dtype=np.float64)
    if idx is None:
        idx, w = topk(logits, k)
    else:
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        w = gate_weights(logits, idx)
    rp = repack(idx, resident)
    sample = np.arange(T) if sample is None else np.asarray(sample, dtype=np.int64)
    pos = np.full(T, -1, dtype=np.int64)
    pos[sample] = np.arange(sample.size)
    out_res = np.zeros((sample.size, H), dtype=np.float64)
    out_off = np.zeros((sample.size, H), dtype=np.float64)
    y_rows = np.full((T * k, H), np.nan, dtype=np.float64) if T * k * H <= (1 << 26) else None
    res = np.asarray(resident, dtype=bool)
    for e in group_order(res):
        c = int(rp["counts"][e])
        if c == 0 or (not offloaded and not res[e]):
            continue
        rows = np.arange(rp["seg_start"][e], rp["seg_start"][e] + c)
        pairs = rp["perm"][rows]
        toks = pairs // k
        keep = pos[toks] >= 0
        if not keep.any():
            continue
        y = expert_ffn(x, toks[keep].astype(np.int32), w13_of(int(e)), w2_of(int(e)))
        if y_rows is not None:
            y_rows[rows[keep]] = y
        dst = out_res if res[e] else out_off
        for r, q in enumerate(pairs[keep]):
            t, j = divmod(int(q), k)
            dst[pos[t]] += w[t, j] * y[r]
    for s in range(n_shared):
        out_res += expert_ffn(x, sample.astype(np.int32), ws13_of(s), ws2_of(s))
    out = dict(rp)
    out.update(logits=logits, idx=idx, w=w, out_res=out_res, out_off=out_off, sample=sample, y_rows=y_rows)
    return out


def gate_weights(logits: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Softmax of each token's scores over a given selection (same rule as ``topk``)."""
    lg = np.asarray(logits, dtype=np.float64)
    sel = np.take_along_axis(lg, np.asarray(idx, dtype=np.int64), axis=1)
    top = sel[:, :1]
    with np.errstate(invalid="ignore"):
        term = np.where(sel == top, 1.0, np.exp(sel - top))
    return term / term.sum(axis=1, keepdims=True)


def layer_forward_synthetic(layer, logits=None, idx=None, sample=None, offloaded=True) -> Dict[str, np.ndarray]:
    """layer_forward on a ``workloads.SyntheticLayer``."""
    c = layer.cfg
    return layer_forward(layer.x, layer.w_router, layer.bias, layer.resident, c.top_k,
                         layer.w13, layer.w2, c.shared, layer.ws13, layer.ws2,
                         logits=logits, idx=idx, sample=sample, offloaded=offloaded)


def near_tie_alternatives(logits: np.ndarray, k: int, delta: float, max_alternatives: int = 16):
    """All top-k selections a rounding of the scores by less than delta/2 could produce.

    For a token whose sorted scores have a gap below ``delta`` among the top k+1,
    both orders of each such adjacent pair are valid outcomes of a top-k taken on
    scores perturbed by less than delta/2.  Returns a dict token -> list of idx
    rows (each a tuple of k expert ids); tokens without a near tie are absent.
    """
    lg = np.asarray(logits, dtype=np.float64)
    T, E = lg.shape
    out = {}
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-lg[t, e], e))
        m = min(E, k + 1)
        head = order[:m]
        close = [abs(lg[t, head[i]] - lg[t, head[i + 1]]) < delta for i in range(m - 1)]
        if not any(close):
            continue
        # blocks of mutually close scores can be ordered in any way
        blocks, cur = [], [head[0]]
        for i in range(m - 1):
            if close[i]:
                cur.append(head[i + 1])
            else:
                blocks.append(cur)
                cur = [head[i + 1]]
        blocks.append(cur)
        # a block that straddles the k boundary may also pull in further tied experts
        tail = order[m:]
        last = blocks[-1]
        for e in tail:
            if abs(lg[t, e] - lg[t, last[-1]]) < delta:
                last.append(e)
            else:
                break
        from itertools import permutations, product
        per_block = []
        for b in blocks:
            per_block.append([tuple(p) for p in permutations(b)][:max_alternatives])
        alts = set()
        for combo in product(*per_block):
            flat = [e for blk in combo for e in blk]
            alts.add(tuple(flat[:k]))
            if len(alts) >= max_alternatives:
                break
        out[t] = sorted(alts)
    return out


# --------------------------------------------------------------------------
# Stage-aware residency (Section IV-C.2) for the stage-structured trace
# --------------------------------------------------------------------------

def stage_plan(log_counts: np.ndarray, n_slots: int, prev_slot: np.ndarray) -> np.ndarray:
    """Residency update at a stage boundary (Section IV-C.2).

    Experts are ranked by their activation count over the completed stage
    (equal counts: lower expert id first); the top n_slots become resident.
    The per-layer slot layout is fixed: an expert that stays resident keeps its
    slot, the least-used incumbents are evicted, and each incoming expert takes
    a freed slot (incoming experts by rank, freed slots by ascending index).
    Returns the new expert -> slot map (-1 = offloaded).
    """
    log = np.asarray(log_counts, dtype=np.int64)
    E = log.size
    ranked = sorted(range(E), key=lambda e: (-int(log[e]), e))
    keep = set(ranked[:n_slots])
    new = np.full(E, -1, dtype=np.int32)
    used = set()
    for e in range(E):
        if prev_slot[e] >= 0 and e in keep:
            new[e] = prev_slot[e]
            used.add(int(prev_slot[e]))
    free = [s for s in range(n_slots) if s not in used]
    incoming = [e for e in ranked[:n_slots] if new[e] < 0]
    for e, s in zip(incoming, free):
        new[e] = s
    return new


def cache_hit_ratio(counts: np.ndarray, resident: np.ndarray) -> float:
    """Fraction of routed pairs whose expert was resident (counts and mask per call, stacked)."""
    c = np.asarray(counts, dtype=np.int64)
    r = np.asarray(resident, dtype=bool)
    tot = int(c.sum())
    return float((c * r).sum()) / tot if tot else 1.0


def stage_replay(counts: np.ndarray, stage_len: np.ndarray, initial_slot: np.ndarray, n_slots: int, lag: int = 0):
    """Stage-aware residency over a decode trace (Sections IV-B.2, IV-C.2, IV-C.3, V-C).

    counts[step, layer, e]: routed pairs per expert of each (step, layer) call;
    routing does not depend on where experts live, so the counts are fixed
    before the policy runs.  A stage's activation log is the sum of its counts
    over all queries in the batch (Section IV-B.2).

    Online policy (the method): stage s runs with the residency planned from the
    log of stage s-1 (the first stage with ``initial_slot``).  Clairvoyant policy
    (the prediction oracle of Section V-C): stage s runs with the residency
    planned from its own log.  CHR = resident pairs / all pairs; eta_CHR is their
    ratio (Eq. upper_bound).

    lag (online policy only): the weights of experts that enter the resident set
    at a boundary are copied to the GPU while the next stage's first steps run
    (Section IV-C.3); for the first ``lag`` steps of every stage after the first,
    only the experts that keep their slot are resident (the evicted ones' slots
    are being overwritten, the incoming ones are still in flight).  lag = 0: the
    new residency holds from the stage's first step.

    Returns slot_history [n_stages, layers, E] (the slots in effect during each
    stage), resident [steps, layers, E], chr_online, chr_clairvoyant, eta_chr.
    """
    c = np.asarray(counts, dtype=np.int64)
    steps, layers, E = c.shape
    ends = np.cumsum(stage_len)
    starts = ends - stage_len
    slot = np.asarray(initial_slot, dtype=np.int32).copy()
    hist = np.empty((len(stage_len), layers, E), dtype=np.int32)
    resident = np.empty((steps, layers, E), dtype=bool)
    hit_on = hit_cv = 0
    prev_res = None
    for s, (a, b) in enumerate(zip(starts, ends)):
        hist[s] = slot
        res = (slot >= 0) & (slot < n_slots)
        resident[a:b] = res[None]
        if s > 0 and lag > 0:
            stay = res & prev_res & (slot == hist[s - 1])    # kept its slot across the boundary
            resident[a:min(a + lag, b)] = stay[None]
        log = c[a:b].sum(axis=0)                     # [layers, E]
        hit_on += int((c[a:b] * resident[a:b]).sum())
        prev_res = res
        for l in range(layers):
            own = stage_plan(log[l], n_slots, np.full(E, -1, np.int32))
            hit_cv += int(log[l][(own >= 0)].sum())
        slot = np.stack([stage_plan(log[l], n_slots, slot[l]) for l in range(layers)])
    total = int(c.sum())
    chr_on = hit_on / total if total else 1.0
    chr_cv = hit_cv / total if total else 1.0
    return {"slot_history": hist, "resident": resident, "chr_online": chr_on, "chr_clairvoyant": chr_cv,
            "eta_chr": chr_on / chr_cv if chr_cv else 1.0}


# --------------------------------------------------------------------------
# Stage-boundary detection (Section IV-B.1)
# --------------------------------------------------------------------------

def cue_matches(cues: Sequence[Sequence[int]], stream: np.ndarray) -> np.ndarray:
    """Transition-cue matches in generated token streams (Section IV-B.1).

    stream[step, b] is the token that sequence b generated at decode step
    `step`; a negative id means no token, and the sequence's window restarts
    there.  After every step the detector checks whether the window of recent
    tokens of each sequence ends with one of the cues (a cue being one or more
    token ids).  Written as that definition: every cue is compared with the
    last tokens of every sequence.  A cue's tokens are never negative, so a
    cue cannot match across a step with no token (nor reach back before the
    first step, padded with -2 below): that is the restart.  Returns [steps, B]
    int32: the id of the longest cue equal to the window's tail after the step
    (identical cues: the lowest id), or -1 when none is.
    """
    s = np.asarray(stream, dtype=np.int64)
    if s.ndim == 1:
        s = s[:, None]
    steps, B = s.shape
    best = np.full((steps, B), -1, dtype=np.int32)
    best_len = np.zeros((steps, B), dtype=np.int64)
    for cid, cue in enumerate(cues):
        c = [int(t) for t in cue]
        L = len(c)
        if L == 0:
            continue
        hit = np.ones((steps, B), dtype=bool)
        for j in range(L):           # token j of the cue sits L-1-j steps back
            back = L - 1 - j
            shifted = np.full((steps, B), -2, dtype=np.int64)
            shifted[back:] = s[:steps - back]
            hit &= shifted == c[j]
        take = hit & (L > best_len)  # longer wins; equal length keeps the earlier (lower) id
        best[take] = cid
        best_len[take] = L
    return best


def stage_lengths_from_events(matched: np.ndarray, steps: int) -> np.ndarray:
    """Stages delimited by detected transitions (Section IV-B.2: one timeline for the batch).

    A cue matched in any sequence at step i ends the current stage with that
    step; the next stage starts at i + 1.  A match at the last step starts no
    stage.  Returns the stage lengths, summing to `steps`.
    """
    m = np.asarray(matched)
    if m.ndim == 1:
        m = m[:, None]
    ev = np.flatnonzero((m[:steps] >= 0).any(axis=1))
    cuts = [int(i) + 1 for i in ev if int(i) + 1 < steps]
    edges = [0] + cuts + [steps]
    return np.diff(np.asarray(edges, dtype=np.int64))


def temporal_coherence(counts: np.ndarray, stage_len: np.ndarray) -> float:
    """TC_seq (Section III, Motivation 2, the TC_seq equation), written as defined.

    R^p[l, e] = tokens of stage p routed to expert e of layer l / tokens layer l
    processed in stage p; sim(R^p, R^{p+1}) = (1/L) sum_l cos(R^p_l, R^{p+1}_l);
    TC_seq = 1/(P-1) sum_{p=1}^{P-1} sim(R^p, R^{p+1}).  counts[step, l, e] are
    routed pairs, and every step processes the same number of tokens in every
    layer, so a layer's tokens in a stage are its pairs / k = its step count x
    batch; the division is done as written even though cosines ignore it.
    NaN for fewer than two stages.
    """
    c = np.asarray(counts, dtype=np.int64)
    steps, L, E = c.shape
    P = len(stage_len)
    if P < 2:
        return float("nan")
    R = []
    a = 0
    for n in stage_len:
        b = a + int(n)
        m = np.zeros((L, E))
        for l in range(L):
            tot = sum(int(c[s, l, e]) for s in range(a, b) for e in range(E))
            for e in range(E):
                m[l, e] = sum(int(c[s, l, e]) for s in range(a, b)) / tot
        R.append(m)
        a = b
    total = 0.0
    for p in range(P - 1):
        sim = 0.0
        for l in range(L):
            u, v = R[p][l], R[p + 1][l]
            dot = sum(u[e] * v[e] for e in range(E))
            nu = sum(u[e] * u[e] for e in range(E)) ** 0.5
            nv = sum(v[e] * v[e] for e in range(E)) ** 0.5
            sim += dot / (nu * nv)
        total += sim / L
    return total / (P - 1)
