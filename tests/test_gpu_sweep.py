"""Seeded sweep of random small layer shapes through the fused forward, against
the oracle (routing, repack and the resident partial output; the same checks as
the fixed edge cases, over shape combinations those do not list).

The shapes cover both FFN paths (T <= 64: streaming kernel; T > 64: tiled kernel
for bf16, the streaming kernel over 64-row chunks for fp32), 0-2 shared experts, partial, empty and full
residency, k up to min(E, 8), and widths that leave ragged tiles."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from test_gpu_parity import run_and_check_layer
from workloads import make_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def moe():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2608_21614_amd as m
    return m


def _shape(i: int):
    rng = np.random.default_rng(1000 + i)
    T = int(rng.choice([1, 3, 8, 17, 31, 32, 40, 64, 65, 96, 150, 200]))
    H = int(rng.choice([64, 128, 192, 256, 512]))
    E = int(rng.choice([2, 5, 8, 16, 33, 64, 100, 256]))
    k = int(rng.integers(1, min(E, 8) + 1))
    F = int(rng.choice([64, 128, 192, 320, 704]))
    S = int(rng.choice([0, 0, 1, 2]))
    Fs = int(rng.choice([64, 256, 576])) if S else 0
    dtype = "f32" if rng.random() < 0.25 else "bf16"
    res = int(rng.choice([0, max(1, E // 3), E // 2, E]))
    return T, H, E, F, k, S, Fs, dtype, res


@pytest.mark.parametrize("i", range(40))
def test_random_shape(moe, i):
    T, H, E, F, k, S, Fs, dtype, res = _shape(i)
    print(f"[case] sweep {i}: T={T} H={H} E={E} F={F} k={k} S={S} Fs={Fs} {dtype} resident={res}", flush=True)
    lay = make_layer(T, H, E, F, k, dtype=dtype, shared=S, shared_ffn=Fs, n_resident=res, residency="random",
                     bias="zipf", seed=77 + i)
    run_and_check_layer(moe, lay)


@pytest.mark.parametrize("i", range(12))
def test_random_shape_hybrid(moe, i):
    """The hybrid layer (offloaded experts on the host, merged by the combine) on random shapes with
    offloaded experts: the full output against the oracle's resident + offloaded sum."""
    from test_gpu_hybrid import run_hybrid
    from gpu_support import TOL
    rng = np.random.default_rng(3000 + i)
    T = int(rng.choice([1, 5, 16, 33, 64, 80]))
    H = int(rng.choice([64, 128, 256]))
    E = int(rng.choice([4, 8, 20, 64]))
    k = int(rng.integers(1, min(E, 8) + 1))
    F = int(rng.choice([64, 128, 320]))
    S = int(rng.choice([0, 1]))
    Fs = 128 if S else 0
    dtype = "f32" if i % 4 == 3 else "bf16"
    res = int(rng.integers(0, E))                       # at least one expert offloaded
    print(f"[case] hybrid sweep {i}: T={T} H={H} E={E} F={F} k={k} S={S} {dtype} resident={res}", flush=True)
    lay = make_layer(T, H, E, F, k, dtype=dtype, shared=S, shared_ffn=Fs, n_resident=res, residency="random",
                     bias="zipf", seed=500 + i)
    err, n_res, _ = run_hybrid(lay, threads=4)
    assert err <= TOL[dtype]
