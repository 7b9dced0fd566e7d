"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI,
compute the oracle's answer on the same seeded inputs, compare.

Comparison rules
* Integer outputs (expert ids, counts, segment starts, permutations, n_res,
  packed offloaded rows) are compared bit-exactly.
* Routing on scores computed by the GPU: every GPU score must be within
  DELTA/2 of the oracle's fp64 score.  Then any token whose top-(k+1) oracle
  scores are all more than DELTA apart has a unique valid routing, which the GPU
  must reproduce exactly.  A token with a closer gap has several valid routings
  (a perturbation below DELTA/2 can reorder it); the oracle enumerates them and
  the GPU's must be one of them; that token's expected output is then the
  oracle's under that routing.
* Given identical scores -- the GPU's own fp32 scores, read back -- the GPU's
  routing equals the oracle's top-k of those scores exactly.
* Router scores: rel-L2 <= 1e-5 against the oracle's fp64 scores.
* Float outputs: rel-L2 over the compared tensor, 1e-5 for fp32 layers and
  1e-2 for bf16 layers with fp32 accumulation.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle

DELTA = 2e-4          # near-tie window of router scores (absolute)
TOL = {"f32": 1e-5, "bf16": 1e-2}
LOGIT_TOL = 1e-5      # rel-L2 of the fp32 router scores against the exact (fp64) scores


def rel_l2(got, ref) -> float:
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    return float(num / den) if den > 0 else float(num)


def row_rel_l2(got, ref) -> np.ndarray:
    """rel-L2 of every row (a diagnostic next to the whole-tensor figure)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref, axis=-1)
    num = np.linalg.norm(got - ref, axis=-1)
    return np.where(den > 0, num / np.where(den > 0, den, 1.0), num)


def host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def expected_routing(lg_ref: np.ndarray, idx_gpu: np.ndarray, k: int):
    """Oracle selection, with near-tied tokens resolved to the GPU's choice if it is a valid one."""
    ref_idx, _ = oracle.topk(lg_ref, k)
    alts = oracle.near_tie_alternatives(lg_ref, k, DELTA)
    exp = ref_idx.copy()
    for t, cands in alts.items():
        g = tuple(int(v) for v in idx_gpu[t])
        assert g in cands, f"token {t}: GPU routing {g} is not a valid near-tie routing {cands}"
        exp[t] = g
    return exp, alts


def check_offloaded_list(x_host: np.ndarray, k: int, perm: np.ndarray, n_res: int, off_rows: np.ndarray,
                         off_w: np.ndarray, w_gpu: np.ndarray):
    P = perm.size
    q = perm[n_res:P]
    np.testing.assert_array_equal(off_rows[: P - n_res], x_host[q // k])
    np.testing.assert_array_equal(off_w[: P - n_res], w_gpu.reshape(-1)[q])
