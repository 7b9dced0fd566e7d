"""Python binding of libsaem_moe.so: one MoE layer's forward on MI355X (gfx950).

Argument marshalling only: every function below validates nothing itself
beyond tensor placement, passes raw device pointers and the current HIP stream
to the C ABI declared in ``include/saem_moe.h``, and raises ``MoeError`` on a
non-OK status.  All computation happens in the library's HIP kernels.  There
is no fallback: importing this package without the built library raises.

Function names are the ABI's.  Shapes and layouts are documented in the header.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsaem_moe.so")

MOE_OK, MOE_ERR_INVALID_ARG, MOE_ERR_UNSUPPORTED, MOE_ERR_WORKSPACE, MOE_ERR_HIP, MOE_ERR_SCRATCH_LIMIT = range(6)
MOE_NOALLOC_SCRATCH_BYTES = 32 << 20
MOE_F32, MOE_BF16 = 0, 1
MOE_LOGITS_IN = 1
MOE_STAGE_EVENTS = 7
MOE_HOST_PIN = 1
MOE_HOST_NO_BF16_DOT = 2

EXPORTED = [
    "moe_abi_version", "moe_status_str", "moe_check_dims", "moe_workspace_bytes", "moe_route_topk",
    "moe_repack", "moe_grouped_ffn", "moe_combine", "moe_layer_forward", "moe_layer_forward_noalloc",
    "moe_stage_accumulate",
    "moe_stage_plan", "moe_pack_weights", "moe_host_ffn", "moe_offload_plan", "moe_read_probe",
    "moe_cue_fsm_words", "moe_cue_build", "moe_cue_step",
]


class MoeError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_str(status)} (status {status})")


class moe_dims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("tokens", "hidden", "experts", "ffn", "top_k", "shared", "shared_ffn", "slots", "dtype")]


_vp = ctypes.c_void_p


class moe_offload_rates(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in
                ("expert_bytes", "flops_per_pair", "link_GBps", "host_GBps", "host_GFLOPs", "gpu_GBps")]


class moe_layer_args(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_size_t), ("dims", moe_dims), ("flags", ctypes.c_uint32),
        ("out_dtype", ctypes.c_int32),
        ("x", _vp), ("w_router", _vp), ("bias", _vp), ("expert_slot", _vp), ("w13", _vp), ("w2", _vp),
        ("ws13", _vp), ("ws2", _vp), ("out", _vp),
        ("logits", _vp), ("topk_idx", _vp), ("topk_w", _vp), ("counts", _vp), ("seg_start", _vp),
        ("perm", _vp), ("inv_perm", _vp), ("n_res", _vp), ("off_rows", _vp), ("off_w", _vp),
        ("stage_events", ctypes.POINTER(ctypes.c_void_p)),
    ]


def _mapped_hip_runtimes() -> set:
    """Paths of every libamdhip64 mapped into this process."""
    paths = set()
    with open("/proc/self/maps") as f:
        for line in f:
            parts = line.split()
            if len(parts) >= 6 and "libamdhip64" in parts[-1]:
                paths.add(os.path.realpath(parts[-1]))
    return paths


def hip_runtime() -> ctypes.CDLL:
    """The HIP runtime this process uses (the one torch loaded)."""
    paths = _mapped_hip_runtimes()
    if len(paths) != 1:
        raise RuntimeError(f"expected exactly one HIP runtime in the process, found {sorted(paths)}")
    return ctypes.CDLL(paths.pop())


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2608_21614_amd/build.py` "
                          "(hipcc, gfx950) before using the HIP path")
    # torch ships its own libamdhip64 (same soname); loading torch first makes the
    # library bind to that copy, so both share one runtime, one set of streams.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    if len(_mapped_hip_runtimes()) != 1:
        raise ImportError(f"two HIP runtimes in one process: {sorted(_mapped_hip_runtimes())}")
    D = ctypes.POINTER(moe_dims)
    i32, u32, sz = ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
    sig = {
        "moe_abi_version": ([], ctypes.c_int),
        "moe_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "moe_check_dims": ([D], ctypes.c_int),
        "moe_workspace_bytes": ([D, ctypes.POINTER(ctypes.c_size_t)], ctypes.c_int),
        "moe_route_topk": ([D, _vp, _vp, _vp, _vp, u32, _vp, _vp, _vp, sz, _vp], ctypes.c_int),
        "moe_repack": ([D, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
        "moe_grouped_ffn": ([D, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, sz, _vp], ctypes.c_int),
        "moe_combine": ([D, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, i32, _vp], ctypes.c_int),
        "moe_layer_forward": ([ctypes.POINTER(moe_layer_args), _vp, sz, _vp], ctypes.c_int),
        "moe_layer_forward_noalloc": ([ctypes.POINTER(moe_layer_args), _vp], ctypes.c_int),
        "moe_stage_accumulate": ([i32, _vp, _vp, _vp], ctypes.c_int),
        "moe_stage_plan": ([i32, i32, _vp, _vp, _vp], ctypes.c_int),
        "moe_pack_weights": ([_vp, _vp, ctypes.c_int64, ctypes.c_int64, i32, _vp], ctypes.c_int),
        "moe_host_ffn": ([D, _vp, _vp, i32, ctypes.POINTER(_vp), ctypes.POINTER(_vp), _vp, _vp, i32, u32],
                         ctypes.c_int),
        "moe_offload_plan": ([i32, _vp, _vp, i32, ctypes.POINTER(moe_offload_rates), i32, _vp], ctypes.c_int),
        "moe_read_probe": ([_vp, ctypes.c_int64, _vp, _vp], ctypes.c_int),
        "moe_cue_fsm_words": ([ctypes.c_int64], ctypes.c_int64),
        "moe_cue_build": ([i32, _vp, _vp, _vp, ctypes.c_int64], ctypes.c_int),
        "moe_cue_step": ([_vp, i32, _vp, _vp, _vp], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


lib = _load()


def status_str(status: int) -> str:
    return lib.moe_status_str(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != MOE_OK:
        raise MoeError(status, where)


def make_dims(tokens: int, hidden: int, experts: int, ffn: int, top_k: int, shared: int = 0, shared_ffn: int = 0,
              slots: int = 0, dtype: int = MOE_BF16) -> moe_dims:
    return moe_dims(tokens, hidden, experts, ffn, top_k, shared, shared_ffn, slots, dtype)


def _p(t) -> Optional[int]:
    """Device pointer of a tensor (or None)."""
    if t is None:
        return None
    if t.device.type != "cuda":
        raise ValueError("libsaem_moe takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libsaem_moe takes contiguous tensors")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def moe_check_dims(dims: moe_dims) -> int:
    return lib.moe_check_dims(ctypes.byref(dims))


def moe_workspace_bytes(dims: moe_dims) -> int:
    n = ctypes.c_size_t(0)
    _check(lib.moe_workspace_bytes(ctypes.byref(dims), ctypes.byref(n)), "moe_workspace_bytes")
    return int(n.value)


def moe_route_topk(dims, x, w_router, bias, logits, topk_idx, topk_w, ws, logits_in: bool = False, stream=None):
    _check(lib.moe_route_topk(ctypes.byref(dims), _p(x), _p(w_router), _p(bias), _p(logits),
                              MOE_LOGITS_IN if logits_in else 0, _p(topk_idx), _p(topk_w), _p(ws),
                              ws.numel() * ws.element_size(), _stream(stream)), "moe_route_topk")


def moe_repack(dims, topk_idx, topk_w, expert_slot, x, counts, seg_start, perm, inv_perm, n_res,
               off_rows=None, off_w=None, stream=None):
    _check(lib.moe_repack(ctypes.byref(dims), _p(topk_idx), _p(topk_w), _p(expert_slot), _p(x), _p(counts),
                          _p(seg_start), _p(perm), _p(inv_perm), _p(n_res), _p(off_rows), _p(off_w),
                          _stream(stream)), "moe_repack")


def moe_grouped_ffn(dims, x, perm, counts, seg_start, expert_slot, w13, w2, ws13, ws2, y, ws, stream=None):
    _check(lib.moe_grouped_ffn(ctypes.byref(dims), _p(x), _p(perm), _p(counts), _p(seg_start), _p(expert_slot),
                               _p(w13), _p(w2), _p(ws13), _p(ws2), _p(y), _p(ws), ws.numel() * ws.element_size(),
                               _stream(stream)), "moe_grouped_ffn")


def moe_combine(dims, topk_idx, topk_w, inv_perm, expert_slot, y, y_off, n_res, out, out_dtype: int, stream=None):
    _check(lib.moe_combine(ctypes.byref(dims), _p(topk_idx), _p(topk_w), _p(inv_perm), _p(expert_slot), _p(y),
                           _p(y_off), _p(n_res), _p(out), int(out_dtype), _stream(stream)), "moe_combine")


def layer_args(dims, x, w_router, bias, expert_slot, w13, w2, ws13, ws2, out, out_dtype: int, flags: int = 0,
               logits=None, topk_idx=None, topk_w=None, counts=None, seg_start=None, perm=None, inv_perm=None,
               n_res=None, off_rows=None, off_w=None, stage_events=None) -> moe_layer_args:
    """Fills a moe_layer_args struct (kept alive by the caller while launches use it).

    stage_events: None, or a ctypes array of MOE_STAGE_EVENTS hipEvent_t handles.
    """
    return moe_layer_args(
        ctypes.sizeof(moe_layer_args), dims, flags, out_dtype, _p(x), _p(w_router), _p(bias), _p(expert_slot),
        _p(w13), _p(w2), _p(ws13), _p(ws2), _p(out), _p(logits), _p(topk_idx), _p(topk_w), _p(counts),
        _p(seg_start), _p(perm), _p(inv_perm), _p(n_res), _p(off_rows), _p(off_w),
        ctypes.cast(stage_events, ctypes.POINTER(ctypes.c_void_p)) if stage_events is not None else None)


def moe_layer_forward(args: moe_layer_args, ws, stream=None):
    _check(lib.moe_layer_forward(ctypes.byref(args), _p(ws), ws.numel() * ws.element_size(), _stream(stream)),
           "moe_layer_forward")


def moe_layer_forward_noalloc(args: moe_layer_args, stream=None):
    """moe_layer_forward on the library's fixed per-GPU scratch array (no workspace, no allocation)."""
    _check(lib.moe_layer_forward_noalloc(ctypes.byref(args), _stream(stream)), "moe_layer_forward_noalloc")


def moe_pack_weights(src, dst, stream=None):
    """Row-major [rows, cols] device matrix -> tile layout (same shape and dtype) in dst."""
    import torch
    if src.shape != dst.shape or src.dtype != dst.dtype or src.dim() < 2:
        raise ValueError("moe_pack_weights: src and dst must have the same [.., rows, cols] shape and dtype")
    dt = MOE_BF16 if src.dtype == torch.bfloat16 else MOE_F32
    rows = src.numel() // src.shape[-1]
    _check(lib.moe_pack_weights(_p(src), _p(dst), rows, src.shape[-1], dt, _stream(stream)), "moe_pack_weights")


def moe_stage_accumulate(experts: int, counts, log, stream=None):
    _check(lib.moe_stage_accumulate(int(experts), _p(counts), _p(log), _stream(stream)), "moe_stage_accumulate")


def moe_read_probe(src, sink, nbytes=None, stream=None):
    """One pass of 16-byte loads over the device tensor `src` (a measurement utility:
    time it on `stream` to get this GPU's streaming-read rate); sink: 1 int32 on the device."""
    n = src.numel() * src.element_size() if nbytes is None else int(nbytes)
    _check(lib.moe_read_probe(_p(src), n, _p(sink), _stream(stream)), "moe_read_probe")


def moe_host_ffn(dims, counts, seg_start, n_res: int, w13_host, w2_host, off_rows, y_off=None, threads: int = 0,
                 pin: bool = False, bf16_dot: bool = True):
    """Host execution of the offloaded experts (host numpy arrays only).

    counts, seg_start: int32 [E]; w13_host[e] / w2_host[e]: row-major [2F, H] / [H, F]
    arrays of the layer dtype (uint16 bf16 bits or float32) for the experts with
    offloaded rows, None for the others; off_rows: [T*k - n_res, H].  Returns
    y_off [T*k - n_res, H] float32 (written into `y_off` when given).  bf16_dot=False keeps
    bf16 layers on the widened fp32 dot products where the CPU has bf16 ones.
    """
    import numpy as np
    E, H = dims.experts, dims.hidden
    cnt = np.ascontiguousarray(counts, dtype=np.int32)
    seg = np.ascontiguousarray(seg_start, dtype=np.int32)
    want = np.uint16 if dims.dtype == MOE_BF16 else np.float32
    n_off = dims.tokens * dims.top_k - int(n_res)
    rows = np.ascontiguousarray(off_rows, dtype=want) if n_off > 0 else None
    if y_off is None:
        y_off = np.empty((max(n_off, 0), H), dtype=np.float32)
    keep = []  # keeps the contiguous weight arrays alive for the call
    p13 = (_vp * E)()
    p2 = (_vp * E)()
    for e in range(E):
        if w13_host[e] is not None:
            a = np.ascontiguousarray(w13_host[e], dtype=want)
            b = np.ascontiguousarray(w2_host[e], dtype=want)
            keep += [a, b]
            p13[e], p2[e] = a.ctypes.data, b.ctypes.data
    _check(lib.moe_host_ffn(ctypes.byref(dims), cnt.ctypes.data, seg.ctypes.data, int(n_res), p13, p2,
                            rows.ctypes.data if rows is not None else None,
                            y_off.ctypes.data if n_off > 0 else None, int(threads),
                            (MOE_HOST_PIN if pin else 0) | (0 if bf16_dot else MOE_HOST_NO_BF16_DOT)),
           "moe_host_ffn")
    return y_off


def moe_offload_plan(counts, expert_slot, slots: int, rates: moe_offload_rates, max_copies: int):
    """Per-expert choice for offloaded experts (host arrays): 1 copy to the GPU, 0 host, -1 resident/idle."""
    import numpy as np
    cnt = np.ascontiguousarray(counts, dtype=np.int32)
    sl = np.ascontiguousarray(expert_slot, dtype=np.int32)
    out = np.empty_like(cnt)
    _check(lib.moe_offload_plan(int(cnt.size), cnt.ctypes.data, sl.ctypes.data, int(slots), ctypes.byref(rates),
                                int(max_copies), out.ctypes.data), "moe_offload_plan")
    return out


def moe_stage_plan(log_host, prev_slot_host, slots: int):
    """Host-side residency plan (numpy int64 log, int32 prev slots) -> numpy int32 new slots."""
    import numpy as np
    log = np.ascontiguousarray(log_host, dtype=np.int64)
    prev = np.ascontiguousarray(prev_slot_host, dtype=np.int32)
    new = np.empty_like(prev)
    _check(lib.moe_stage_plan(int(log.size), int(slots), log.ctypes.data, prev.ctypes.data, new.ctypes.data),
           "moe_stage_plan")
    return new


def moe_cue_build(cues):
    """Stage-boundary cue machine (Section IV-B.1) from a list of token-id sequences -> numpy int32 words."""
    import numpy as np
    seqs = [np.asarray(c, dtype=np.int64).ravel() for c in cues]
    off = np.zeros(len(seqs) + 1, dtype=np.int32)
    if seqs:
        off[1:] = np.cumsum([len(c) for c in seqs])
    toks = (np.concatenate(seqs) if seqs else np.zeros(0)).astype(np.int32)
    words = int(lib.moe_cue_fsm_words(int(off[-1])))
    fsm = np.zeros(max(words, 1), dtype=np.int32)
    _check(lib.moe_cue_build(len(seqs), off.ctypes.data, toks.ctypes.data, fsm.ctypes.data, words), "moe_cue_build")
    return fsm


def moe_cue_step(fsm, tokens, state):
    """Feeds one token per sequence (numpy int32 [B]); updates `state` in place -> matched cue ids [B] (-1: none)."""
    import numpy as np
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    if state.dtype != np.int32 or not state.flags.c_contiguous or state.shape != tok.shape:
        raise ValueError("state must be a C-contiguous int32 array shaped like tokens")
    matched = np.empty_like(tok)
    _check(lib.moe_cue_step(fsm.ctypes.data, int(tok.size), tok.ctypes.data, state.ctypes.data, matched.ctypes.data),
           "moe_cue_step")
    return matched
