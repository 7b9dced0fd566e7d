// kernels.hpp -- internal launch interface between the C ABI (abi.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace saem {

// Shapes of one layer, already validated by the ABI.
struct Shape {
    int T, H, E, F, k, S, Fs, slots;
    int bf16;  // 1: bf16 activations and weights, 0: fp32
};

// Decode batches (T <= 64) route through K-sliced partial scores: the number of
// slices (0 for larger batches); their scratch is [slices][64][E] fp32.
bool front_small_fits(const Shape& s);
int router_slices(const Shape& s);

// Router scores + top-k gate.  part: scratch of router_slices(s) * 64 * E floats.
hipError_t launch_route_topk(const Shape& s, const void* x, const void* w_router, const float* bias, float* logits,
                             bool logits_in, int32_t* topk_idx, float* topk_w, float* part, hipStream_t st);

// Expert-aligned repacking: histogram, group-order scan, stable permutation,
// residency split (one workgroup).
hipError_t launch_repack(const Shape& s, const int32_t* topk_idx, const int32_t* expert_slot, int32_t* counts,
                         int32_t* seg_start, int32_t* perm, int32_t* inv_perm, int32_t* n_res, hipStream_t st);

// Packs the rows of the offloaded pairs: off_rows[p - n_res] = x[perm[p] / k], off_w[p - n_res] = w[perm[p]].
hipError_t launch_offload_pack(const Shape& s, const void* x, const float* topk_w, const int32_t* perm,
                               const int32_t* n_res, void* off_rows, float* off_w, hipStream_t st);

// Grouped SwiGLU FFN.  Row space: packed rows [0, T*k) then shared rows T*k + s*T + t.
struct FfnArgs {
    const void* x;
    const int32_t* perm;
    const int32_t* counts;
    const int32_t* seg_start;
    const int32_t* expert_slot;
    const void* w13;
    const void* w2;
    const void* ws13;
    const void* ws2;
    void* act;          // [rows, Fa] activation dtype: silu(x W1) * (x W3)
    int Fa;             // row stride of act = max(F, Fs)
    float* y;           // [ks][rows][H] fp32 partial sums over K chunks of the down projection
    int ks;             // number of K chunks of the down projection
    long long y_ks_stride;
    // optional: pack the offloaded rows in extra workgroups (of phase 1 at decode,
    // of the token gather at bf16 prefill)
    const float* topk_w = nullptr;
    const int32_t* n_res = nullptr;
    void* off_rows = nullptr;
    float* off_w = nullptr;
    // bf16 prefill: the token rows gathered into the MFMA tile layout, ffn_gather_rows(s) x H,
    // and the tiled kernels' item tables (ffn_tile_meta_bytes(s), 32-byte aligned)
    void* xg = nullptr;
    int32_t* tmeta = nullptr;
    // bf16 prefill: phase 2 writes the expert outputs here in bf16 ([rows][H]) instead of y
    void* y16 = nullptr;
    // decode (ffn_fuses_repack): phase 1 takes the repacking over from topk_idx. Its
    // workgroups derive their groups from the ids, one more workgroup writes counts,
    // seg_start, perm, inv_perm and n_res (which phase 2 and the combine read), and the
    // offloaded rows are packed by workgroups of phase 2
    const int32_t* topk_idx = nullptr;
    int32_t* rp_counts = nullptr;
    int32_t* rp_seg_start = nullptr;
    int32_t* rp_perm = nullptr;
    int32_t* rp_inv_perm = nullptr;
    int32_t* rp_n_res = nullptr;
};

// True when the fused forward leaves the repacking to FFN phase 1 (decode batches).
bool ffn_fuses_repack(const Shape& s);

// True when the expert outputs are bf16 (y16) rather than fp32 partial sums (y).
bool ffn_y_bf16(const Shape& s);
// Bytes of the expert-output buffer: bf16 rows, or ks fp32 chunks of rows.
size_t ffn_y_bytes(const Shape& s);

// Rows of the activation buffer (row stride Fa; the bf16 prefill path pads every
// group to 16 rows) and of the gathered-token buffer (0: the path has none).
long long ffn_act_rows(const Shape& s);
long long ffn_gather_rows(const Shape& s);
size_t ffn_tile_meta_bytes(const Shape& s);

// bf16 prefill: gathers the resident groups' token rows (and the batch in order,
// for the shared experts) into a.xg, and packs the offloaded rows if asked;
// must precede launch_grouped_ffn on the stream.  No-op on the other paths.
hipError_t launch_gather_tokens(const Shape& s, const FfnArgs& a, hipStream_t st);

// True when the FFN path packs the offloaded rows itself (in phase 1 at decode,
// in the token gather at bf16 prefill).
bool ffn_packs_offloaded(const Shape& s);

// Number of K chunks the down projection is split into (1 = direct sums).
int ffn_down_splits(const Shape& s);
// Launches phase 1 then phase 2; records `between` (if not null) after phase 1.
hipError_t launch_grouped_ffn(const Shape& s, const FfnArgs& a, hipStream_t st, hipEvent_t between = nullptr);

// y_out[p] = sum_c y[c][p] for the resident packed rows and the shared rows (y_bf16:
// one chunk of bf16 rows, widened to fp32).
hipError_t launch_reduce_splits(const Shape& s, const int32_t* counts, const int32_t* expert_slot, const void* y,
                                bool y_bf16, int ks, long long y_ks_stride, float* y_out, hipStream_t st);

// Deterministic combine back to token order.  y: ks fp32 chunks, or (y_bf16) one chunk of bf16 rows.
hipError_t launch_combine(const Shape& s, const int32_t* topk_idx, const float* topk_w, const int32_t* inv_perm,
                          const int32_t* expert_slot, const void* y, bool y_bf16, int ks, long long y_ks_stride,
                          const float* y_off, const int32_t* n_res, void* out, bool out_bf16, hipStream_t st);

// Row-major [rows, K] -> tile layout.
hipError_t launch_pack_weights(const void* src, void* dst, long long rows, long long K, bool bf16, hipStream_t st);

hipError_t launch_stage_accumulate(int E, const int32_t* counts, int64_t* log, hipStream_t st);

// Measurement utility: one pass of 16-byte loads over `bytes` of src (a multiple of 16).
hipError_t launch_read_probe(const void* src, long long bytes, uint32_t* sink, hipStream_t st);

}  // namespace saem
