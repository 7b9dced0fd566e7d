"""Seeded synthetic MoE-layer workloads.

This module only draws random inputs with the shapes, value distributions and
routing structure of the five MoE-layer workloads (a tiny fp32 layer, a
Mixtral-like decode layer, a fine-grained shared+routed decode layer, a
prefill chunk, and a stage-structured decode trace) and one GPU's share of a
layer under expert parallelism (``ExpertShard``, a view).  It holds none of the
layer's arithmetic: no router product, no top-k, no repacking, no expert FFN,
no combine.  Both the CPU oracle's tests and the GPU path's tests and bench
consume the buffers it returns, so both sides see bit-identical inputs.

Storage layouts are the ones the C ABI takes (K-contiguous):

* ``x``         [T, H]        activations
* ``w_router``  [E, H]        router weight, row e scores expert e
* ``bias``      [E] fp32      additive router bias (or ``None``)
* ``w13(e)``    [2F, H]       rows 0..F-1 are the gate projection W1 (one row
                              per output feature), rows F..2F-1 the up
                              projection W3
* ``w2(e)``     [H, F]        row h is output feature h of the down projection
* ``ws13(s)``, ``ws2(s)``     the same for shared expert s with Fs features

bf16 tensors are numpy ``uint16`` arrays holding bf16 bit patterns, rounded
from fp32 draws with round-to-nearest-even.  fp32 tensors are ``float32``.

Every tensor is drawn from its own counter-keyed PCG64 stream
(``SeedSequence(seed, spawn_key=(layer, tag, index, chunk))``), so a tensor's
values do not depend on which other tensors were generated, in which order,
or on how many threads drew them.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field, replace
from typing import Dict, Optional

import numpy as np

__all__ = [
    "MoEConfig", "TraceConfig", "CONFIGS", "TRACE", "SyntheticLayer", "StageTrace",
    "bf16_bits_to_f32", "f32_to_bf16_bits", "make_layer", "ExpertShard",
]

# tags of the per-tensor random streams
_TAG_X, _TAG_WR, _TAG_W13, _TAG_W2, _TAG_WS13, _TAG_WS2 = 1, 2, 3, 4, 5, 6
_TAG_BIAS, _TAG_RES, _TAG_SLOT, _TAG_STAGE, _TAG_DIR = 7, 8, 9, 10, 11
_TAG_CUE, _TAG_TOK, _TAG_PLANT = 12, 13, 14

_CHUNK = 1 << 22  # elements per independent stream chunk
_THREADS = max(1, min(16, int(os.environ.get("MOE_GEN_THREADS", os.cpu_count() or 1))))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even) -> uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).copy()
    u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (u >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(seed, spawn_key=tuple(int(k) for k in key)))


def _normal(seed: int, key: tuple, shape, std: float, dtype: str) -> np.ndarray:
    """N(0, std^2) draws, fp32, optionally rounded to bf16 bits; chunked streams."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.uint16 if dtype == "bf16" else np.float32)
    nchunks = max(1, (n + _CHUNK - 1) // _CHUNK)

    def work(c: int) -> None:
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        if hi <= lo:
            return
        a = _rng(seed, *key, c).standard_normal(hi - lo, dtype=np.float32)
        a *= np.float32(std)
        if dtype == "bf16":
            u = a.view(np.uint32)
            u += np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
            u >>= np.uint32(16)
            out[lo:hi] = u
        else:
            out[lo:hi] = a

    if nchunks == 1 or _THREADS == 1:
        for c in range(nchunks):
            work(c)
    else:
        with ThreadPoolExecutor(min(_THREADS, nchunks)) as ex:
            list(ex.map(work, range(nchunks)))
    return out.reshape(shape)


@dataclass(frozen=True)
class MoEConfig:
    """Shape and structure of one synthetic MoE layer."""
    name: str
    dtype: str              # "f32" or "bf16": activations, router and expert weights
    tokens: int             # T
    hidden: int             # H
    experts: int            # E routed experts
    ffn: int                # F, per routed expert
    top_k: int              # k
    shared: int = 0         # S always-on shared experts
    shared_ffn: int = 0     # Fs
    n_resident: int = 0     # routed experts resident on the GPU (ECR = n_resident / E)
    residency: str = "all"  # "all" | "random" (seeded) | "zipf_top" (hottest by popularity)
    bias: str = "none"      # "none" | "zipf"
    zipf_s: float = 1.1
    x_std: float = 1.0
    w_std: float = 0.02
    description: str = ""

    def logit_std(self) -> float:
        """Standard deviation of one router score x.w_e for N(0,x_std) x, N(0,w_std) w."""
        return self.x_std * self.w_std * math.sqrt(self.hidden)


CONFIGS: Dict[str, MoEConfig] = {
    "c1_tiny_f32": MoEConfig(
        "c1_tiny_f32", "f32", tokens=16, hidden=256, experts=8, ffn=512, top_k=2,
        n_resident=8, residency="all",
        description="tiny fp32 MoE layer, 16 tokens, H 256, 8 SwiGLU experts F 512, top-2, all resident"),
    "c2_mixtral_decode": MoEConfig(
        "c2_mixtral_decode", "bf16", tokens=32, hidden=4096, experts=8, ffn=14336, top_k=2,
        n_resident=4, residency="random",
        description="Mixtral-style bf16 decode batch of 32 tokens, H 4096, 8 experts F 14336, top-2, 4/8 resident"),
    "c3_shared_decode": MoEConfig(
        "c3_shared_decode", "bf16", tokens=64, hidden=2048, experts=60, ffn=1408, top_k=4,
        shared=1, shared_ffn=5632, n_resident=30, residency="zipf_top", bias="zipf",
        description="fine-grained bf16 decode batch of 64 tokens, H 2048, 60 routed F 1408 top-4 + 1 shared F 5632, 30/60 resident, Zipf(1.1)"),
    "c4_prefill": MoEConfig(
        "c4_prefill", "bf16", tokens=2048, hidden=2048, experts=64, ffn=1408, top_k=6,
        shared=2, shared_ffn=1408, n_resident=48, residency="zipf_top", bias="zipf",
        description="bf16 prefill chunk of 2048 tokens, H 2048, 64 routed F 1408 top-6 + 2 shared F 1408, 48/64 resident, Zipf(1.1)"),
    # the prefill shape in fp32: the fp32 path (MFMA 16x16x4) at prefill size
    "c4_prefill_f32": MoEConfig(
        "c4_prefill_f32", "f32", tokens=2048, hidden=2048, experts=64, ffn=1408, top_k=6,
        shared=2, shared_ffn=1408, n_resident=48, residency="zipf_top", bias="zipf",
        description="fp32 prefill chunk of 2048 tokens, H 2048, 64 routed F 1408 top-6 + 2 shared F 1408, 48/64 resident, Zipf(1.1)"),
    # many small experts with a wide top-k (the Qwen3-MoE family the paper evaluates): the
    # shape of the bookkeeping A/B, where per-expert launches cost the most
    "c6_qwen3_decode": MoEConfig(
        "c6_qwen3_decode", "bf16", tokens=64, hidden=2048, experts=128, ffn=768, top_k=8,
        n_resident=64, residency="zipf_top", bias="zipf",
        description="Qwen3-MoE-like bf16 decode batch of 64 tokens, H 2048, 128 experts F 768, top-8, 64/128 resident, Zipf(1.1)"),
}


@dataclass(frozen=True)
class TraceConfig:
    """Stage-structured decode trace: stacked Mixtral-style layers, per-stage router bias."""
    name: str = "c5_stage_trace"
    layers: int = 8
    steps: int = 2048
    batch: int = 16
    hidden: int = 4096
    experts: int = 8
    ffn: int = 14336
    top_k: int = 2
    n_slots: int = 2                 # resident experts per layer (25% ECR)
    dirichlet_alpha: float = 0.3
    mean_stage_len: float = 256.0
    # 0: every (stage, layer) popularity is an independent draw; rho > 0: stage s's
    # popularity is rho x stage s-1's + (1 - rho) x a fresh draw (more coherent stages)
    stage_persistence: float = 0.0
    x_std: float = 1.0
    w_std: float = 0.02
    dtype: str = "bf16"
    # generated-token stream of the batch with transition cues at the stage boundaries
    vocab: int = 32000
    n_cues: int = 12
    max_cue_len: int = 4
    token_zipf_s: float = 1.1
    cue_min_rank: int = 1000        # cue tokens are drawn from popularity ranks >= this

    def layer_config(self) -> MoEConfig:
        return MoEConfig(self.name, self.dtype, tokens=self.batch, hidden=self.hidden,
                         experts=self.experts, ffn=self.ffn, top_k=self.top_k,
                         n_resident=self.n_slots, residency="random", bias="none",
                         x_std=self.x_std, w_std=self.w_std,
                         description=f"one layer call of the stage trace: {self.dtype} decode batch of {self.batch} "
                                     f"tokens, H {self.hidden}, {self.experts} experts F {self.ffn}, top-{self.top_k}, "
                                     f"{self.n_slots}/{self.experts} resident")

    def logit_std(self) -> float:
        return self.x_std * self.w_std * math.sqrt(self.hidden)


TRACE = TraceConfig()


def _gumbel_scale(logit_std: float) -> float:
    """Scale that maps a normal score of the given std onto the Gumbel(0,1) std pi/sqrt(6).

    With bias b_e = scale * ln p_e, the perturbed argmax of (score + bias) picks
    expert e with probability close to p_e (the Gumbel-max construction).
    """
    return logit_std * math.sqrt(6.0) / math.pi


class SyntheticLayer:
    """One seeded MoE layer.  Expert weights are generated lazily and cached."""

    def __init__(self, cfg: MoEConfig, seed: int = 0, layer: int = 0,
                 tokens: Optional[int] = None, cache_weights: bool = True):
        self.cfg = cfg if tokens is None else replace(cfg, tokens=tokens)
        self.seed = int(seed)
        self.layer = int(layer)
        self.cache_weights = cache_weights
        c = self.cfg
        self._w: Dict[tuple, np.ndarray] = {}
        self.x = _normal(seed, (layer, _TAG_X, 0), (c.tokens, c.hidden), c.x_std, c.dtype)
        self.w_router = _normal(seed, (layer, _TAG_WR, 0), (c.experts, c.hidden), c.w_std, c.dtype)
        # popularity ranks: a seeded permutation, rank[e] in 1..E
        self.popularity_rank = _rng(seed, layer, _TAG_BIAS, 0).permutation(c.experts) + 1
        if c.bias == "zipf":
            p = self.popularity_rank.astype(np.float64) ** (-c.zipf_s)
            p /= p.sum()
            self.bias = (_gumbel_scale(c.logit_std()) * np.log(p)).astype(np.float32)
        else:
            self.bias = None
        self.resident = self._draw_residency()
        self.expert_slot = self._assign_slots(self.resident)

    # residency map: expert -> slot (or -1 = offloaded)
    def _draw_residency(self) -> np.ndarray:
        c = self.cfg
        res = np.zeros(c.experts, dtype=bool)
        if c.residency == "all":
            res[:] = True
        elif c.residency == "random":
            res[_rng(self.seed, self.layer, _TAG_RES, 0).choice(c.experts, c.n_resident, replace=False)] = True
        elif c.residency == "zipf_top":
            res[self.popularity_rank <= c.n_resident] = True
        else:
            raise ValueError(f"unknown residency {c.residency!r}")
        return res

    def _assign_slots(self, resident: np.ndarray) -> np.ndarray:
        """Resident experts get slots 0..n-1 in a seeded order; offloaded experts get -1."""
        slot = np.full(self.cfg.experts, -1, dtype=np.int32)
        ids = np.flatnonzero(resident)
        order = _rng(self.seed, self.layer, _TAG_SLOT, 0).permutation(len(ids))
        slot[ids] = order.astype(np.int32)
        return slot

    def set_residency(self, resident: np.ndarray, expert_slot: Optional[np.ndarray] = None) -> None:
        self.resident = np.asarray(resident, dtype=bool).copy()
        self.expert_slot = (self._assign_slots(self.resident) if expert_slot is None
                            else np.asarray(expert_slot, dtype=np.int32).copy())

    @property
    def n_slots(self) -> int:
        return int(self.resident.sum())

    def _get(self, tag: int, idx: int, shape) -> np.ndarray:
        key = (tag, idx)
        if key in self._w:
            return self._w[key]
        a = _normal(self.seed, (self.layer, tag, idx), shape, self.cfg.w_std, self.cfg.dtype)
        if self.cache_weights:
            self._w[key] = a
        return a

    def w13(self, e: int) -> np.ndarray:
        c = self.cfg
        return self._get(_TAG_W13, e, (2 * c.ffn, c.hidden))

    def w2(self, e: int) -> np.ndarray:
        c = self.cfg
        return self._get(_TAG_W2, e, (c.hidden, c.ffn))

    def ws13(self, s: int) -> np.ndarray:
        c = self.cfg
        return self._get(_TAG_WS13, s, (2 * c.shared_ffn, c.hidden))

    def ws2(self, s: int) -> np.ndarray:
        c = self.cfg
        return self._get(_TAG_WS2, s, (c.hidden, c.shared_ffn))

    def drop_cache(self) -> None:
        self._w.clear()

    def slot_experts(self) -> np.ndarray:
        """Expert id held by each slot, slot order."""
        out = np.empty(self.n_slots, dtype=np.int32)
        for e in np.flatnonzero(self.resident):
            out[self.expert_slot[e]] = e
        return out


class ExpertShard:
    """One GPU's share of a layer under n-way expert parallelism (a view: no tensor is redrawn).

    Routing is replicated, so every shard sees the layer's own ``x``, router and bias and
    computes the same top-k.  The routed experts are split into n contiguous id blocks
    (sizes as ``numpy.array_split`` gives them); shard g holds block g in slots 0.. (id
    order) and marks every other expert absent.  Each shared expert is split by its FFN
    columns in 64-column units (the SwiGLU acts on each column on its own, so the shards'
    partial outputs add up to the whole layer's); a shard whose share of the columns is
    empty holds no shared expert.
    """

    def __init__(self, layer: "SyntheticLayer", n: int, g: int):
        c = layer.cfg
        if not (n >= 1 and 0 <= g < n):
            raise ValueError(f"shard {g} of {n}")
        self.layer = layer
        self.n, self.g = int(n), int(g)
        ids = np.array_split(np.arange(c.experts), n)[g]
        self.expert_ids = ids.astype(np.int32)
        self.expert_slot = np.full(c.experts, -1, dtype=np.int32)
        self.expert_slot[ids] = np.arange(len(ids), dtype=np.int32)
        self.resident = self.expert_slot >= 0
        f0 = f1 = 0
        if c.shared > 0:
            if c.shared_ffn % 64:
                raise ValueError("shared FFN width must be a multiple of 64")
            units = np.array_split(np.arange(c.shared_ffn // 64), n)[g]
            if len(units):
                f0, f1 = int(units[0]) * 64, (int(units[-1]) + 1) * 64
        self.shared_cols = (f0, f1)
        self.cfg = replace(c, shared=c.shared if f1 > f0 else 0, shared_ffn=f1 - f0, n_resident=len(ids),
                           description=f"{c.description}; expert-parallel shard {g} of {n}: routed experts "
                                       f"{f'[{int(ids[0])}, {int(ids[-1]) + 1})' if len(ids) else 'none'}, "
                                       f"shared columns [{f0}, {f1})")
        self.x, self.w_router, self.bias = layer.x, layer.w_router, layer.bias

    @property
    def n_slots(self) -> int:
        return len(self.expert_ids)

    def slot_experts(self) -> np.ndarray:
        return self.expert_ids.copy()

    def w13(self, e: int) -> np.ndarray:
        return self.layer.w13(e)

    def w2(self, e: int) -> np.ndarray:
        return self.layer.w2(e)

    def ws13(self, s: int) -> np.ndarray:
        f0, f1 = self.shared_cols
        F = self.layer.cfg.shared_ffn
        w = self.layer.ws13(s)
        return np.ascontiguousarray(np.concatenate([w[f0:f1], w[F + f0:F + f1]]))

    def ws2(self, s: int) -> np.ndarray:
        f0, f1 = self.shared_cols
        return np.ascontiguousarray(self.layer.ws2(s)[:, f0:f1])


def make_layer(tokens: int, hidden: int, experts: int, ffn: int, top_k: int, dtype: str = "bf16",
               shared: int = 0, shared_ffn: int = 0, n_resident: Optional[int] = None,
               residency: str = "random", bias: str = "none", seed: int = 0,
               x_std: float = 1.0, w_std: float = 0.02) -> SyntheticLayer:
    """A layer of arbitrary shape (edge cases, ragged tails)."""
    if n_resident is None:
        n_resident = experts
        residency = "all"
    cfg = MoEConfig("custom", dtype, tokens, hidden, experts, ffn, top_k, shared, shared_ffn,
                    n_resident, residency, bias, x_std=x_std, w_std=w_std)
    return SyntheticLayer(cfg, seed)


@dataclass
class StageTrace:
    """Stage structure of the decode trace: stage lengths and per-(stage, layer) router bias.

    Stage lengths are Geometric(1/mean) on {1, 2, ...}, drawn until they cover
    all steps (the last stage is truncated).  Each (stage, layer) gets a
    popularity vector p ~ Dirichlet(alpha), clamped at 1e-6, mapped to a router
    bias b = scale * ln p with the Gumbel-matching scale.  Every (step, layer)
    call sees a fresh N(0,1) activation batch.  Initial residency per layer is a
    seeded random choice of n_slots experts.
    """
    cfg: TraceConfig
    seed: int = 0
    stage_len: np.ndarray = field(init=False)
    stage_bias: np.ndarray = field(init=False)      # [n_stages, layers, E] fp32
    initial_resident: np.ndarray = field(init=False)  # [layers, E] bool

    def __post_init__(self) -> None:
        c = self.cfg
        rng = _rng(self.seed, 0, _TAG_STAGE, 0)
        lens = []
        total = 0
        while total < c.steps:
            n = int(rng.geometric(1.0 / c.mean_stage_len))
            n = min(n, c.steps - total)
            lens.append(n)
            total += n
        self.stage_len = np.asarray(lens, dtype=np.int64)
        scale = _gumbel_scale(c.logit_std())
        bias = np.empty((len(lens), c.layers, c.experts), dtype=np.float32)
        prev = [None] * c.layers
        for s in range(len(lens)):
            for l in range(c.layers):
                p = _rng(self.seed, l, _TAG_DIR, s).dirichlet(np.full(c.experts, c.dirichlet_alpha))
                if c.stage_persistence > 0 and prev[l] is not None:
                    p = c.stage_persistence * prev[l] + (1.0 - c.stage_persistence) * p
                prev[l] = p
                p = np.maximum(p, 1e-6)
                bias[s, l] = (scale * np.log(p)).astype(np.float32)
        self.stage_bias = bias
        res = np.zeros((c.layers, c.experts), dtype=bool)
        for l in range(c.layers):
            res[l, _rng(self.seed, l, _TAG_RES, 0).choice(c.experts, c.n_slots, replace=False)] = True
        self.initial_resident = res

    @property
    def n_stages(self) -> int:
        return len(self.stage_len)

    def stage_of_step(self) -> np.ndarray:
        return np.repeat(np.arange(self.n_stages), self.stage_len)

    def stage_ends(self) -> np.ndarray:
        """Step index at which each stage ends (inclusive)."""
        return np.cumsum(self.stage_len) - 1

    def x(self, step: int, layer: int) -> np.ndarray:
        c = self.cfg
        return _normal(self.seed, (layer, _TAG_X, 1 + step), (c.batch, c.hidden), c.x_std, c.dtype)

    def cues(self) -> list:
        """Synthetic transition cues: n_cues token-id sequences of 1..max_cue_len tokens.

        They stand in for a model's cue phrases ("Alternatively", "On second
        thought", ...) split into subword tokens; the first cue has one token so
        that every boundary can take a cue.  Tokens come from the less popular
        part of the vocabulary (ranks >= cue_min_rank of the background's Zipf
        order), so background text completes a cue only now and then.
        """
        c = self.cfg
        rng = _rng(self.seed, 0, _TAG_CUE, 0)
        order = self._token_order()
        out = []
        for i in range(c.n_cues):
            n = 1 if i == 0 else int(rng.integers(1, c.max_cue_len + 1))
            ranks = rng.integers(c.cue_min_rank, c.vocab, size=n)
            out.append([int(order[r]) for r in ranks])
        return out

    def _token_order(self) -> np.ndarray:
        """Token id of each popularity rank (a seeded permutation of the vocabulary)."""
        return _rng(self.seed, 0, _TAG_TOK, 0).permutation(self.cfg.vocab)

    def token_stream(self) -> dict:
        """Generated tokens of the batch, [steps, batch] int32, with the cues planted at the boundaries.

        Background tokens are Zipf(token_zipf_s) over the vocabulary.  For every
        stage after the first, one sequence (seeded, among those whose last
        planted cue ends before this one starts, so no cue overwrites another)
        generates a cue whose last token falls on the last step of the previous
        stage, so a detector that matches cues sees the transition exactly at
        the planted boundary.  Returns stream, cues and planted (the step of
        each planted cue's last token).
        """
        c = self.cfg
        steps, B = c.steps, c.batch
        order = self._token_order()
        p = np.arange(1, c.vocab + 1, dtype=np.float64) ** (-c.token_zipf_s)
        p /= p.sum()
        ranks = _rng(self.seed, 0, _TAG_TOK, 1).choice(c.vocab, size=(steps, B), p=p)
        stream = order[ranks].astype(np.int32)
        cues = self.cues()
        rng = _rng(self.seed, 0, _TAG_PLANT, 0)
        planted = []
        last_end = np.full(B, -1, dtype=np.int64)      # step of each sequence's last planted token
        for a in np.cumsum(self.stage_len)[:-1]:
            a = int(a)
            fits = [i for i, q in enumerate(cues) if len(q) <= a]
            q = cues[fits[int(rng.integers(len(fits)))]]
            free = np.flatnonzero(last_end < a - len(q))
            if free.size == 0:     # boundaries too close for this cue: the one-token cue always fits
                q = cues[0]
                free = np.flatnonzero(last_end < a - 1)
            b = int(free[int(rng.integers(free.size))])
            stream[a - len(q):a, b] = q
            last_end[b] = a - 1
            planted.append(a - 1)
        return {"stream": stream, "cues": cues, "planted": np.asarray(planted, dtype=np.int64)}

    def layer(self, layer: int, cache_weights: bool = True) -> SyntheticLayer:
        """The layer's weights (router, experts); x and bias are per call."""
        lay = SyntheticLayer(self.cfg.layer_config(), self.seed, layer=layer, cache_weights=cache_weights)
        lay.set_residency(self.initial_resident[layer])
        return lay
