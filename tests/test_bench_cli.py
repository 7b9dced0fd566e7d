"""Host-side parts of bench.py: the one-GPU contract, the algorithmic byte and
FLOP accounting behind `roofline`, and the stale-counter guard (CPU only)."""
from __future__ import annotations

import json
import os
import subprocess
import sys
from dataclasses import replace

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads import CONFIGS  # noqa: E402


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=300, cwd=ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"] or "one MI355X" in line["error"]


def test_algorithmic_bytes_by_hand():
    """c2-like: 4 resident experts of which 3 are active; b = 2 bytes."""
    cfg = CONFIGS["c2_mixtral_decode"]
    T, H, E, F, k = cfg.tokens, cfg.hidden, cfg.experts, cfg.ffn, cfg.top_k
    resident = np.array([1, 0, 1, 0, 1, 0, 1, 0], bool)
    counts = np.array([10, 20, 0, 5, 9, 11, 9, 0])          # sums to T * k = 64
    assert counts.sum() == T * k
    a = bench.algorithmic_bytes(cfg, counts, resident)
    assert a["active"] == 3                                   # expert 2 is resident but idle
    assert a["n_res"] == 10 + 0 + 9 + 9 and a["n_off"] == 64 - 28
    assert a["phase1_bytes"] == 3 * 2 * H * F * 2 + T * H * 2
    assert a["expert_weight_bytes"] == 3 * 3 * H * F * 2
    assert a["flops"] == 6 * H * F * 28 + 2 * T * H * E
    assert a["phase1_flops"] == 4 * H * F * 28
    assert a["layer_bytes"] == (3 * 3 * H * F * 2 + H * E * 2 + 2 * T * H * 2 + 36 * H * 2 + T * k * 16)


def test_algorithmic_bytes_count_shared_experts():
    cfg = replace(CONFIGS["c3_shared_decode"], experts=4, top_k=2, tokens=8)
    H, F, Fs = cfg.hidden, cfg.ffn, cfg.shared_ffn
    a = bench.algorithmic_bytes(cfg, np.array([4, 4, 4, 4]), np.array([1, 1, 0, 0], bool))
    assert a["active"] == 2 and a["n_res"] == 8
    assert a["phase1_bytes"] == 2 * 2 * H * F * 2 + 2 * H * Fs * 2 + 8 * H * 2
    assert a["flops"] == 6 * H * F * 8 + 6 * H * Fs * 8 + 2 * 8 * H * 4


def test_traffic_is_null_when_the_kernel_source_changed(tmp_path, monkeypatch):
    text = ("workload: wl\nkernel: k\nsource_sha: {sha}\ntraffic_bytes_per_launch: 123456\n")
    (tmp_path / "traffic_ffn_phase1_wl.txt").write_text(text.format(sha=bench.kernel_source_hash()))
    monkeypatch.setattr(bench, "TRAFFIC_DIR", str(tmp_path))
    assert bench.read_traffic("wl") == 123456.0
    (tmp_path / "traffic_ffn_phase1_wl.txt").write_text(text.format(sha="0000000000000000"))
    assert bench.read_traffic("wl") is None
    assert bench.read_traffic("missing") is None


@pytest.mark.parametrize("workload", ["c2_mixtral_decode", "c3_shared_decode", "c4_prefill", "c5_stage_trace",
                                      "c6_qwen3_decode"])
def test_committed_traffic_matches_the_current_kernels(workload):
    """The committed counter summaries were taken with the FFN sources as they are now."""
    assert bench.read_traffic(workload) is not None, f"profiles/traffic_ffn_phase1_{workload}.txt is stale or missing"


def test_layer_roofline_takes_the_fp32_peak_for_fp32_layers():
    alg = {"layer_bytes": 8e12 * 10e-6, "flops": 157.3e12 * 50e-6}   # 10 us of bytes, 50 us of fp32 flops
    r = bench.layer_roofline(alg, ms_per_step=0.1, dtype="f32")
    assert r["bound"] == "mfma" and abs(r["t_roof_us"] - 50.0) < 1e-9 and abs(r["frac"] - 0.5) < 1e-12


def test_layer_roofline_bound_and_fraction():
    alg = {"layer_bytes": 8e12 * 100e-6, "flops": 2.5e15 * 40e-6}     # 100 us of bytes, 40 us of flops
    r = bench.layer_roofline(alg, ms_per_step=0.2)
    assert r["bound"] == "hbm" and abs(r["t_roof_us"] - 100.0) < 1e-9 and abs(r["frac"] - 0.5) < 1e-12
    alg = {"layer_bytes": 8e12 * 10e-6, "flops": 2.5e15 * 50e-6}
    r = bench.layer_roofline(alg, ms_per_step=0.1)
    assert r["bound"] == "mfma" and abs(r["t_roof_us"] - 50.0) < 1e-9 and abs(r["frac"] - 0.5) < 1e-12
