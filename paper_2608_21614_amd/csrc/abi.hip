// abi.hip -- the C ABI of libsaem_moe.so: argument checks, workspace layout and
// launch sequencing of the device calls.  Every check runs on the host before
// anything is enqueued and never touches device memory; the shape rules
// (moe_check_dims) and the other host-only calls are in host_abi.cpp.
#include <string.h>

#include <algorithm>
#include <mutex>

#include "../../include/saem_moe.h"
#include "kernels.hpp"

// Workspace of moe_layer_forward_noalloc: one fixed array per GPU, held until the
// process ends.  Host code never passes `scratch` itself to a kernel (on the
// host it names a stand-in, not device memory): it looks up the array's device
// address once per device and passes that.
static __device__ __align__(256) unsigned char scratch[MOE_NOALLOC_SCRATCH_BYTES];

namespace {

using saem::Shape;

// Arrays read or written with 16-byte vector accesses (activations, weights,
// outputs, workspace) must be 16-byte aligned; index, count and gate arrays only
// need their element alignment (4 bytes; 8 for the int64 stage log).
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }
bool ok_ptr(const void* p) { return p != nullptr && aligned16(p); }
bool ok_opt(const void* p) { return p == nullptr || aligned16(p); }
// A required vector array: non-NULL and aligned, except that an array with no elements may be NULL.
bool ok_arr(const void* p, long long n) { return n == 0 ? aligned16(p) : ok_ptr(p); }
// The same for 4-byte element arrays.
bool ok_ptr4(const void* p) { return p != nullptr && aligned4(p); }
bool ok_opt4(const void* p) { return p == nullptr || aligned4(p); }
bool ok_arr4(const void* p, long long n) { return n == 0 ? aligned4(p) : ok_ptr4(p); }

Shape shape_of(const moe_dims* d) {
    Shape s;
    s.T = d->tokens;
    s.H = d->hidden;
    s.E = d->experts;
    s.F = d->ffn;
    s.k = d->top_k;
    s.S = d->shared;
    s.Fs = d->shared > 0 ? d->shared_ffn : 0;
    s.slots = d->slots;
    s.bf16 = d->dtype == MOE_BF16 ? 1 : 0;
    return s;
}

// Workspace layout (256-byte aligned regions).
struct Layout {
    size_t logits, idx, w, counts, seg, nres, perm, inv, part, act, xg, meta, y, total;
    int ks, Fa;
    long long rows;
};

size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

Layout layout_of(const Shape& s) {
    Layout L;
    const size_t T = s.T, E = s.E, k = s.k, H = s.H;
    L.rows = (long long)s.T * s.k + (long long)s.S * s.T;
    L.Fa = std::max(s.F, s.Fs);
    L.ks = saem::ffn_down_splits(s);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align256(off + std::max<size_t>(bytes, 1));
        return at;
    };
    L.logits = take(T * E * 4);
    L.idx = take(T * k * 4);
    L.w = take(T * k * 4);
    L.counts = take(E * 4);
    L.seg = take(E * 4);
    L.nres = take(4);
    L.perm = take(T * k * 4);
    L.inv = take(T * k * 4);
    L.part = take((size_t)saem::router_slices(s) * 64 * E * 4);
    L.act = take((size_t)saem::ffn_act_rows(s) * L.Fa * (s.bf16 ? 2 : 4));
    L.xg = take((size_t)saem::ffn_gather_rows(s) * H * 2);
    L.meta = take(saem::ffn_tile_meta_bytes(s));
    L.y = take(saem::ffn_y_bytes(s));
    L.total = off;
    return L;
}

template <typename T>
T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

moe_status hip_status(hipError_t e) { return e == hipSuccess ? MOE_OK : MOE_ERR_HIP; }

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array, looked up on the first
// call on that device.  *out stays NULL when the stream belongs to another device
// (the array would not be that device's).
hipError_t scratch_for_stream(hipStream_t st, void** out) {
    *out = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(st, &sdev);
    if (e != hipSuccess) return e;
    if (sdev != dev || dev < 0 || dev >= kMaxDevices) return hipSuccess;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" {



moe_status moe_workspace_bytes(const moe_dims* dims, size_t* bytes) {
    const moe_status st = moe_check_dims(dims);
    if (st != MOE_OK) return st;
    if (!bytes) return MOE_ERR_INVALID_ARG;
    *bytes = layout_of(shape_of(dims)).total;
    return MOE_OK;
}

moe_status moe_route_topk(const moe_dims* dims, const void* x, const void* w_router, const float* bias,
                          float* logits, uint32_t flags, int32_t* topk_idx, float* topk_w, void* ws, size_t ws_bytes,
                          void* stream) {
    moe_status st = moe_check_dims(dims);
    if (st != MOE_OK) return st;
    if (flags & ~MOE_LOGITS_IN) return MOE_ERR_INVALID_ARG;
    const bool lin = (flags & MOE_LOGITS_IN) != 0;
    const long long T = dims->tokens;
    if (!ok_arr4(logits, T) || !ok_arr4(topk_idx, T) || !ok_arr4(topk_w, T)) return MOE_ERR_INVALID_ARG;
    if (!lin && (!ok_arr(x, T) || !ok_ptr(w_router) || !ok_opt4(bias))) return MOE_ERR_INVALID_ARG;
    const Shape s = shape_of(dims);
    const Layout L = layout_of(s);
    if (!ws || ws_bytes < L.total || !aligned16(ws)) return MOE_ERR_WORKSPACE;
    return hip_status(saem::launch_route_topk(s, x, w_router, lin ? nullptr : bias, logits, lin, topk_idx, topk_w,
                                              at<float>(ws, L.part), static_cast<hipStream_t>(stream)));
}

moe_status moe_repack(const moe_dims* dims, const int32_t* topk_idx, const float* topk_w,
                      const int32_t* expert_slot, const void* x, int32_t* counts, int32_t* seg_start,
                      int32_t* perm, int32_t* inv_perm, int32_t* n_res, void* off_rows, float* off_w,
                      void* stream) {
    moe_status st = moe_check_dims(dims);
    if (st != MOE_OK) return st;
    const long long T = dims->tokens;
    if (!ok_arr4(topk_idx, T) || !ok_ptr4(expert_slot) || !ok_ptr4(counts) || !ok_ptr4(seg_start) ||
        !ok_arr4(perm, T) || !ok_arr4(inv_perm, T) || !ok_ptr4(n_res) || !ok_opt(off_rows) || !ok_opt4(off_w))
        return MOE_ERR_INVALID_ARG;
    if (off_rows && !ok_arr(x, T)) return MOE_ERR_INVALID_ARG;
    if (off_w && !ok_arr4(topk_w, T)) return MOE_ERR_INVALID_ARG;
    const Shape s = shape_of(dims);
    hipStream_t hs = static_cast<hipStream_t>(stream);
    hipError_t e = saem::launch_repack(s, topk_idx, expert_slot, counts, seg_start, perm, inv_perm, n_res, hs);
    if (e == hipSuccess) e = saem::launch_offload_pack(s, x, topk_w, perm, n_res, off_rows, off_w, hs);
    return hip_status(e);
}

moe_status moe_grouped_ffn(const moe_dims* dims, const void* x, const int32_t* perm, const int32_t* counts,
                           const int32_t* seg_start, const int32_t* expert_slot, const void* w13, const void* w2,
                           const void* ws13, const void* ws2, float* y, void* ws, size_t ws_bytes, void* stream) {
    moe_status st = moe_check_dims(dims);
    if (st != MOE_OK) return st;
    const long long T = dims->tokens;
    if (!ok_arr(x, T) || !ok_arr4(perm, T) || !ok_ptr4(counts) || !ok_ptr4(seg_start) || !ok_ptr4(expert_slot) ||
        !ok_arr(y, T))
        return MOE_ERR_INVALID_ARG;
    if (dims->slots > 0 && (!ok_ptr(w13) || !ok_ptr(w2))) return MOE_ERR_INVALID_ARG;
    if (dims->shared > 0 && (!ok_ptr(ws13) || !ok_ptr(ws2))) return MOE_ERR_INVALID_ARG;
    const Shape s = shape_of(dims);
    const Layout L = layout_of(s);
    if (!ws || ws_bytes < L.total || !aligned16(ws)) return MOE_ERR_WORKSPACE;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    saem::FfnArgs a;
    a.x = x; a.perm = perm; a.counts = counts; a.seg_start = seg_start; a.expert_slot = expert_slot;
    a.w13 = w13; a.w2 = w2; a.ws13 = ws13; a.ws2 = ws2;
    a.act = at<char>(ws, L.act);
    a.xg = at<char>(ws, L.xg);
    a.tmeta = at<int32_t>(ws, L.meta);
    a.Fa = L.Fa;
    a.ks = L.ks;
    a.y_ks_stride = L.rows * (long long)s.H;
    // the expert outputs go straight to y unless they are split-K partial sums or bf16 rows,
    // which are added (widened) into y afterwards, resident and shared rows only
    const bool y16 = saem::ffn_y_bf16(s);
    a.y = (L.ks == 1 && !y16) ? y : at<float>(ws, L.y);
    a.y16 = y16 ? at<char>(ws, L.y) : nullptr;
    hipError_t e = saem::launch_gather_tokens(s, a, hs);
    if (e == hipSuccess) e = saem::launch_grouped_ffn(s, a, hs);
    if (e == hipSuccess && (L.ks > 1 || y16))
        e = saem::launch_reduce_splits(s, counts, expert_slot, y16 ? a.y16 : a.y, y16, L.ks, a.y_ks_stride, y, hs);
    return hip_status(e);
}

moe_status moe_combine(const moe_dims* dims, const int32_t* topk_idx, const float* topk_w,
                       const int32_t* inv_perm, const int32_t* expert_slot, const float* y,
                       const float* y_off, const int32_t* n_res, void* out, int32_t out_dtype, void* stream) {
    moe_status st = moe_check_dims(dims);
    if (st != MOE_OK) return st;
    if (out_dtype != MOE_F32 && out_dtype != MOE_BF16) return MOE_ERR_INVALID_ARG;
    const long long T = dims->tokens;
    if (!ok_arr4(topk_idx, T) || !ok_arr4(topk_w, T) || !ok_arr4(inv_perm, T) || !ok_ptr4(expert_slot) ||
        !ok_arr(y, T) || !ok_arr(out, T) || !ok_opt(y_off))
        return MOE_ERR_INVALID_ARG;
    if (y_off && !ok_ptr4(n_res)) return MOE_ERR_INVALID_ARG;
    const Shape s = shape_of(dims);
    return hip_status(saem::launch_combine(s, topk_idx, topk_w, inv_perm, expert_slot, y, false, 1, 0, y_off,
                                           y_off ? n_res : nullptr,
                                           out, out_dtype == MOE_BF16, static_cast<hipStream_t>(stream)));
}

// The fused forward on a given workspace; moe_layer_forward and moe_layer_forward_noalloc
// (the library's fixed scratch array) both run it.
static moe_status layer_forward(const moe_layer_args* a, void* ws, size_t ws_bytes, hipStream_t hs) {
    if (!a || a->struct_size != sizeof(moe_layer_args)) return MOE_ERR_INVALID_ARG;
    const moe_dims* d = &a->dims;
    moe_status st = moe_check_dims(d);
    if (st != MOE_OK) return st;
    if (a->flags & ~MOE_LOGITS_IN) return MOE_ERR_INVALID_ARG;
    if (a->out_dtype != MOE_F32 && a->out_dtype != MOE_BF16) return MOE_ERR_INVALID_ARG;
    const bool lin = (a->flags & MOE_LOGITS_IN) != 0;
    const long long T = d->tokens;
    if (!ok_arr(a->x, T) || !ok_ptr4(a->expert_slot) || !ok_arr(a->out, T)) return MOE_ERR_INVALID_ARG;
    if (!lin && (!ok_ptr(a->w_router) || !ok_opt4(a->bias))) return MOE_ERR_INVALID_ARG;
    if (lin && !ok_arr4(a->logits, T)) return MOE_ERR_INVALID_ARG;
    if (d->slots > 0 && (!ok_ptr(a->w13) || !ok_ptr(a->w2))) return MOE_ERR_INVALID_ARG;
    if (d->shared > 0 && (!ok_ptr(a->ws13) || !ok_ptr(a->ws2))) return MOE_ERR_INVALID_ARG;
    if (!ok_opt4(a->logits) || !ok_opt4(a->topk_idx) || !ok_opt4(a->topk_w) || !ok_opt4(a->counts) ||
        !ok_opt4(a->seg_start) || !ok_opt4(a->perm) || !ok_opt4(a->inv_perm) || !ok_opt4(a->n_res) ||
        !ok_opt(a->off_rows) || !ok_opt4(a->off_w))
        return MOE_ERR_INVALID_ARG;
    const Shape s = shape_of(d);
    const Layout L = layout_of(s);
    if (!ws || ws_bytes < L.total || !aligned16(ws)) return MOE_ERR_WORKSPACE;

    float* logits = a->logits ? a->logits : at<float>(ws, L.logits);
    int32_t* idx = a->topk_idx ? a->topk_idx : at<int32_t>(ws, L.idx);
    float* w = a->topk_w ? a->topk_w : at<float>(ws, L.w);
    int32_t* counts = a->counts ? a->counts : at<int32_t>(ws, L.counts);
    int32_t* seg = a->seg_start ? a->seg_start : at<int32_t>(ws, L.seg);
    int32_t* perm = a->perm ? a->perm : at<int32_t>(ws, L.perm);
    int32_t* inv = a->inv_perm ? a->inv_perm : at<int32_t>(ws, L.inv);
    int32_t* nres = a->n_res ? a->n_res : at<int32_t>(ws, L.nres);

    hipEvent_t ev[MOE_STAGE_EVENTS] = {};
    if (a->stage_events)
        for (int i = 0; i < MOE_STAGE_EVENTS; ++i) ev[i] = static_cast<hipEvent_t>(a->stage_events[i]);
    auto mark = [&](hipError_t e, int i) {
        if (e == hipSuccess && ev[i]) e = hipEventRecord(ev[i], hs);
        return e;
    };

    hipError_t e = mark(hipSuccess, 0);
    if (e == hipSuccess)
        e = mark(saem::launch_route_topk(s, a->x, a->w_router, lin ? nullptr : a->bias, logits, lin, idx, w,
                                         at<float>(ws, L.part), hs),
                 1);
    // decode: FFN phase 1 does the repacking itself (one launch fewer); the stage event
    // after the repack then follows the routing directly
    const bool fuse_repack = saem::ffn_fuses_repack(s);
    if (e == hipSuccess)
        e = mark(fuse_repack ? hipSuccess
                             : saem::launch_repack(s, idx, a->expert_slot, counts, seg, perm, inv, nres, hs),
                 2);
    if (s.T == 0) {
        for (int i = 3; i < MOE_STAGE_EVENTS && e == hipSuccess; ++i) e = mark(hipSuccess, i);
        return hip_status(e);
    }
    const bool fold_pack = saem::ffn_packs_offloaded(s);
    saem::FfnArgs f;
    if (fold_pack) {
        f.topk_w = w;
        f.n_res = nres;
        f.off_rows = a->off_rows;
        f.off_w = a->off_w;
    }
    f.x = a->x; f.perm = perm; f.counts = counts; f.seg_start = seg; f.expert_slot = a->expert_slot;
    if (fuse_repack) {
        f.topk_idx = idx;
        f.rp_counts = counts;
        f.rp_seg_start = seg;
        f.rp_perm = perm;
        f.rp_inv_perm = inv;
        f.rp_n_res = nres;
    }
    f.w13 = a->w13; f.w2 = a->w2; f.ws13 = a->ws13; f.ws2 = a->ws2;
    f.act = at<char>(ws, L.act);
    f.xg = at<char>(ws, L.xg);
    f.tmeta = at<int32_t>(ws, L.meta);
    f.Fa = L.Fa;
    const bool y16 = saem::ffn_y_bf16(s);
    f.y = at<float>(ws, L.y);
    f.y16 = y16 ? at<char>(ws, L.y) : nullptr;
    f.ks = L.ks;
    f.y_ks_stride = L.rows * (long long)s.H;
    // the token gather of the bf16 prefill path (with the offloaded-row pack), or the
    // standalone pack of the fp32 prefill path; at decode the pack is in FFN phase 2
    if (e == hipSuccess)
        e = mark(fold_pack ? saem::launch_gather_tokens(s, f, hs)
                           : saem::launch_offload_pack(s, a->x, w, perm, nres, a->off_rows, a->off_w, hs), 3);
    if (e == hipSuccess) e = mark(saem::launch_grouped_ffn(s, f, hs, ev[4]), 5);
    if (e == hipSuccess)
        e = mark(saem::launch_combine(s, idx, w, inv, a->expert_slot, at<char>(ws, L.y), y16, L.ks, f.y_ks_stride,
                                      nullptr, nres,
                                      a->out, a->out_dtype == MOE_BF16, hs), 6);
    return hip_status(e);
}

moe_status moe_layer_forward(const moe_layer_args* a, void* ws, size_t ws_bytes, void* stream) {
    return layer_forward(a, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

moe_status moe_layer_forward_noalloc(const moe_layer_args* a, void* stream) {
    if (!a || a->struct_size != sizeof(moe_layer_args)) return MOE_ERR_INVALID_ARG;
    const moe_status st = moe_check_dims(&a->dims);
    if (st != MOE_OK) return st;
    if (layout_of(shape_of(&a->dims)).total > MOE_NOALLOC_SCRATCH_BYTES) return MOE_ERR_SCRATCH_LIMIT;
    hipStream_t hs = static_cast<hipStream_t>(stream);
    void* ws = nullptr;
    if (scratch_for_stream(hs, &ws) != hipSuccess) return MOE_ERR_HIP;
    if (!ws) return MOE_ERR_INVALID_ARG;  // the stream is not on the current device
    return layer_forward(a, ws, MOE_NOALLOC_SCRATCH_BYTES, hs);
}

moe_status moe_pack_weights(const void* src, void* dst, int64_t rows, int64_t cols, int32_t dtype, void* stream) {
    if (dtype != MOE_F32 && dtype != MOE_BF16) return MOE_ERR_INVALID_ARG;
    if (rows < 0 || cols < 0) return MOE_ERR_INVALID_ARG;
    if (rows % 16 != 0 || cols % 32 != 0) return MOE_ERR_UNSUPPORTED;
    const long long n = (long long)rows * cols;
    if (!ok_arr(src, n) || !ok_arr(dst, n)) return MOE_ERR_INVALID_ARG;
    const size_t bytes = (size_t)n * (dtype == MOE_BF16 ? 2 : 4);
    const uintptr_t s0 = reinterpret_cast<uintptr_t>(src), d0 = reinterpret_cast<uintptr_t>(dst);
    if (n > 0 && s0 < d0 + bytes && d0 < s0 + bytes) return MOE_ERR_INVALID_ARG;  // overlapping buffers
    return hip_status(
        saem::launch_pack_weights(src, dst, rows, cols, dtype == MOE_BF16, static_cast<hipStream_t>(stream)));
}

moe_status moe_stage_accumulate(int32_t experts, const int32_t* counts, int64_t* log, void* stream) {
    if (experts <= 0 || experts > 256 || !ok_ptr4(counts) || !log || (reinterpret_cast<uintptr_t>(log) & 7u))
        return MOE_ERR_INVALID_ARG;
    return hip_status(saem::launch_stage_accumulate(experts, counts, log, static_cast<hipStream_t>(stream)));
}

moe_status moe_read_probe(const void* src, int64_t bytes, uint32_t* sink, void* stream) {
    if (bytes < 0 || bytes % 16 != 0 || (bytes > 0 && !ok_ptr(src)) || !ok_ptr4(sink)) return MOE_ERR_INVALID_ARG;
    return hip_status(saem::launch_read_probe(src, bytes, sink, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
