"""Concurrent layer calls from several host threads, each on its own stream with its own workspace.

The ABI allows calls on distinct streams with distinct workspaces to run at the
same time: the library keeps no device or host state between calls, and a call
writes only its outputs and its workspace.  Three threads start together and
each enqueues eight layer calls on its own stream without synchronising in
between:
  * a bf16 decode layer with a shared expert and offloaded experts,
  * the same layer's weights (read by both at once) on another input batch,
    with a second workspace,
  * a bf16 prefill layer.
Every output must equal the same call made alone, bit for bit (the path is
deterministic).
"""
from __future__ import annotations

import threading

import numpy as np
import pytest
import torch

from workloads import make_layer

pytestmark = pytest.mark.gpu

NAMES = ("out", "logits", "topk_idx", "topk_w", "counts", "seg_start", "n_res")


def say(*a):
    print("[concurrency]", *a, flush=True)


def _bits(t: torch.Tensor) -> torch.Tensor:
    return t.contiguous().view(torch.uint8)


def test_threads_on_own_streams_and_workspaces_match_serial_calls():
    import paper_2608_21614_amd as moe
    from paper_2608_21614_amd.device import DeviceLayer, to_device

    dec = make_layer(40, 256, 16, 512, 4, "bf16", shared=1, shared_ffn=256, n_resident=10, residency="random",
                     bias="zipf", seed=5)
    pre = make_layer(130, 256, 8, 256, 2, "bf16", n_resident=6, residency="random", seed=6)
    d_dec, d_pre = DeviceLayer(dec), DeviceLayer(pre)
    ws2 = torch.empty_like(d_dec.ws)
    x2 = to_device(np.ascontiguousarray(dec.x[::-1]))

    # (layer, workspace, input or None) per thread
    jobs = [(d_dec, d_dec.ws, None), (d_dec, ws2, x2), (d_pre, d_pre.ws, None)]
    say("decode T 40, same weights on a second input, prefill T 130")

    refs = []
    for dev, ws, x in jobs:                     # each call alone
        o = dev.alloc_outputs()
        moe.moe_layer_forward(dev.args(o, x=x), ws)
        torch.cuda.synchronize()
        refs.append(o)
    assert not torch.equal(refs[0]["logits"], refs[1]["logits"])

    outs = [dev.alloc_outputs() for dev, _, _ in jobs]
    for o in outs:                              # garbage the calls must overwrite
        for t in o.values():
            if isinstance(t, torch.Tensor):
                _bits(t).fill_(0x5A)
    streams = [torch.cuda.Stream() for _ in jobs]
    torch.cuda.synchronize()
    start = threading.Barrier(len(jobs))
    errors = []

    def run(i):
        dev, ws, x = jobs[i]
        try:
            args = dev.args(outs[i], x=x)
            start.wait(timeout=60)
            for _ in range(8):
                moe.moe_layer_forward(args, ws, streams[i])
            streams[i].synchronize()
        except Exception as exc:                # reported on the main thread
            errors.append((i, repr(exc)))

    threads = [threading.Thread(target=run, args=(i,)) for i in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a thread did not finish"
    assert not errors, errors
    torch.cuda.synchronize()
    for i, (o, ref) in enumerate(zip(outs, refs)):
        for name in NAMES:
            assert torch.equal(_bits(o[name]), _bits(ref[name])), f"thread {i}: {name}"
        P = int(o["topk_idx"].numel())
        for name in ("perm", "inv_perm"):
            assert torch.equal(o[name][:P], ref[name][:P]), f"thread {i}: {name}"
        say(f"  thread {i}: eight calls identical to the call made alone")
