// combine.hip -- merge of the expert outputs back to token order
// (SAEM Section IV-D.2).  A gather in a fixed order, with no atomics, so two
// runs give bitwise-identical outputs; the paper's atomic accumulation is not
// reproducible (Section V-C).
//
// Workgroup = one token x 1024 hidden columns (4 per thread, 16-byte loads of fp32
// expert outputs; 2048 columns, 8 per thread, when they come in bf16):
//   acc = 0  (fp32)
//   for j in 0..k-1:  acc += w[t,j] * (sum_c y[c][inv[t,j]])          resident
//                     acc += w[t,j] * y_off[inv[t,j] - n_res]          offloaded, if given
//   for s in 0..S-1:  acc += sum_c y[c][T*k + s*T + t]
//   out[t] = round(acc)
#include "common.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

// sum_c y[c][row, h..h+3] over the ks K chunks, in chunk order; all loads issued first.
__device__ __forceinline__ f32x4 sum_chunks(const float* __restrict__ y, int ks, long long stride, size_t off) {
    constexpr int kMax = 16;
    f32x4 p[kMax];
#pragma unroll
    for (int c = 0; c < kMax; ++c)
        if (c < ks) p[c] = *reinterpret_cast<const f32x4*>(y + c * stride + off);
    f32x4 v = p[0];
#pragma unroll
    for (int c = 1; c < kMax; ++c)
        if (c < ks) v += p[c];
    return v;
}

// Workgroup = one token x 1024 columns.  The token's indices (choices, gate
// weights, packed rows, residency) are loaded first, all at once; then every
// contribution's loads are issued without branches (a contribution that does
// not apply reads a valid row and is replaced by zero, never multiplied by it);
// then the sums run in the fixed order above.  KS >= ks is the compile-time
// bound on the K chunks; above two chunks the loads go one contribution at a
// time (all of its chunks together), which keeps the registers in bounds.
template <bool kOutBf16, int KS>
__global__ void __launch_bounds__(256)
    k_combine(int T, int H, int E, int k, int S, int slots, const int32_t* __restrict__ topk_idx,
              const float* __restrict__ topk_w, const int32_t* __restrict__ inv_perm,
              const int32_t* __restrict__ expert_slot, const float* __restrict__ y, int ks, long long stride,
              const float* __restrict__ y_off, const int32_t* __restrict__ n_res_p, void* __restrict__ out) {
    constexpr int kK = 8, kS = 8;  // bounds on k and S (the ABI checks both)
    const int t = blockIdx.x;
    const int h = (blockIdx.y * 256 + threadIdx.x) * 4;
    if (h >= H) return;
    const int P = T * k;
    // with n_res at hand, a choice is resident iff its packed row lies in the resident
    // prefix [0, n_res) (the repacking puts resident pairs first), which spares a round
    // trip to expert_slot
    const int nres = n_res_p ? *n_res_p : 0;

    // the token's choices
    int e[kK], p[kK];
    float w[kK];
#pragma unroll
    for (int j = 0; j < kK; ++j) {
        e[j] = -1;
        p[j] = -1;
        w[j] = 0.f;
        if (j < k) {
            e[j] = topk_idx[t * k + j];
            p[j] = inv_perm[t * k + j];
            w[j] = topk_w[t * k + j];
        }
    }
    // where each choice's row lives: 1 = y (resident), 2 = y_off (offloaded, given), 0 = nowhere
    int src[kK];
#pragma unroll
    for (int j = 0; j < kK; ++j) {
        src[j] = 0;
        if (j < k && e[j] >= 0 && e[j] < E && p[j] >= 0 && p[j] < P) {
            const bool res = n_res_p ? p[j] < nres : is_resident(expert_slot[e[j]], slots);
            if (res) src[j] = 1;
            else if (y_off && p[j] >= nres) src[j] = 2;
        }
    }
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    f32x4 acc = zero;
    if constexpr (KS <= 2) {
        // every contribution's loads at once, then the fixed-order sums
        f32x4 v[kK][KS], vs[kS][KS];
#pragma unroll
        for (int j = 0; j < kK; ++j) {
            const size_t off = (size_t)(src[j] ? p[j] : 0) * H + h;
            const float* base = (src[j] == 2) ? y_off + (off - (size_t)nres * H) : y + off;
#pragma unroll
            for (int c = 0; c < KS; ++c) {
                const bool use = src[j] == 1 ? c < ks : (src[j] == 2 && c == 0);
                const f32x4 l = *reinterpret_cast<const f32x4*>(base + (use ? c * stride : 0));
                v[j][c] = use ? l : zero;
            }
        }
#pragma unroll
        for (int s2 = 0; s2 < kS; ++s2) {
            const size_t off = (size_t)(s2 < S ? P + s2 * T + t : 0) * H + h;
#pragma unroll
            for (int c = 0; c < KS; ++c) {
                const bool use = s2 < S && c < ks;
                const f32x4 l = *reinterpret_cast<const f32x4*>(y + off + (use ? c * stride : 0));
                vs[s2][c] = use ? l : zero;
            }
        }
#pragma unroll
        for (int j = 0; j < kK; ++j) {
            if (!src[j]) continue;  // uniform over the workgroup
            f32x4 r = v[j][0];
            if (KS > 1 && src[j] == 1 && ks > 1) r += v[j][KS - 1];
            acc += w[j] * r;
        }
#pragma unroll
        for (int s2 = 0; s2 < kS; ++s2) {
            if (s2 >= S) continue;
            f32x4 r = vs[s2][0];
            if (KS > 1 && ks > 1) r += vs[s2][KS - 1];
            acc += r;
        }
    } else {
        // one contribution at a time, its chunk loads together
        for (int j = 0; j < k; ++j) {
            if (src[j] == 1) acc += w[j] * sum_chunks(y, ks, stride, (size_t)p[j] * H + h);
            else if (src[j] == 2) acc += w[j] * *reinterpret_cast<const f32x4*>(y_off + (size_t)(p[j] - nres) * H + h);
        }
        for (int s2 = 0; s2 < S; ++s2) acc += sum_chunks(y, ks, stride, ((size_t)P + (size_t)s2 * T + t) * H + h);
    }
    if (kOutBf16) {
        u32x2 packed;
        packed.x = pack_bf16x2(acc.x, acc.y);
        packed.y = pack_bf16x2(acc.z, acc.w);
        *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(out) + (size_t)t * H + h) = packed;
    } else {
        *reinterpret_cast<f32x4*>(static_cast<float*>(out) + (size_t)t * H + h) = acc;
    }
}

// The same merge when the expert outputs come in bf16 (one chunk): 8 columns per
// thread, so that every row load is 16 bytes; workgroup = one token x 2048 columns.
// kOff: the caller gave the offloaded rows' outputs (y_off); without them the kernel
// holds no registers for those rows.
template <bool kOutBf16, bool kOff>
__global__ void __launch_bounds__(256)
    k_combine_y16(int T, int H, int E, int k, int S, int slots, const int32_t* __restrict__ topk_idx,
                  const float* __restrict__ topk_w, const int32_t* __restrict__ inv_perm,
                  const int32_t* __restrict__ expert_slot, const uint16_t* __restrict__ y16,
                  const float* __restrict__ y_off, const int32_t* __restrict__ n_res_p, void* __restrict__ out) {
    constexpr int kK = 8, kS = 8;  // bounds on k and S (the ABI checks both)
    const int t = blockIdx.x;
    const int h = (blockIdx.y * 256 + threadIdx.x) * 8;
    if (h >= H) return;
    const int P = T * k;
    const int nres = n_res_p ? *n_res_p : 0;
    int e[kK], p[kK];
    float w[kK];
#pragma unroll
    for (int j = 0; j < kK; ++j) {
        e[j] = -1;
        p[j] = -1;
        w[j] = 0.f;
        if (j < k) {
            e[j] = topk_idx[t * k + j];
            p[j] = inv_perm[t * k + j];
            w[j] = topk_w[t * k + j];
        }
    }
    int src[kK];  // 1 = y16 (resident), 2 = y_off (offloaded, given), 0 = nowhere
#pragma unroll
    for (int j = 0; j < kK; ++j) {
        src[j] = 0;
        if (j < k && e[j] >= 0 && e[j] < E && p[j] >= 0 && p[j] < P) {
            const bool res = n_res_p ? p[j] < nres : is_resident(expert_slot[e[j]], slots);
            if (res) src[j] = 1;
            else if (kOff && p[j] >= nres) src[j] = 2;
        }
    }
    // every load first (a contribution that does not apply reads row 0 and is dropped)
    u32x4 v[kK], vs[kS];
    f32x4 vo[kK][2];
#pragma unroll
    for (int j = 0; j < kK; ++j) {
        const size_t off = (size_t)(src[j] == 1 ? p[j] : 0) * H + h;
        v[j] = *reinterpret_cast<const u32x4*>(y16 + off);
        if (kOff && src[j] == 2) {
            const float* r = y_off + (size_t)(p[j] - nres) * H + h;
            vo[j][0] = *reinterpret_cast<const f32x4*>(r);
            vo[j][1] = *reinterpret_cast<const f32x4*>(r + 4);
        }
    }
#pragma unroll
    for (int s2 = 0; s2 < kS; ++s2)
        vs[s2] = *reinterpret_cast<const u32x4*>(y16 + (size_t)(s2 < S ? P + s2 * T + t : 0) * H + h);
    const f32x4 zero = {0.f, 0.f, 0.f, 0.f};
    f32x4 lo = zero, hi = zero;
#pragma unroll
    for (int j = 0; j < kK; ++j) {
        if (src[j] == 1) {
            lo += w[j] * bf16x4_to_f32(u32x2{v[j].x, v[j].y});
            hi += w[j] * bf16x4_to_f32(u32x2{v[j].z, v[j].w});
        } else if (kOff && src[j] == 2) {
            lo += w[j] * vo[j][0];
            hi += w[j] * vo[j][1];
        }
    }
#pragma unroll
    for (int s2 = 0; s2 < kS; ++s2) {
        if (s2 >= S) continue;
        lo += bf16x4_to_f32(u32x2{vs[s2].x, vs[s2].y});
        hi += bf16x4_to_f32(u32x2{vs[s2].z, vs[s2].w});
    }
    if (kOutBf16) {
        u32x4 packed;
        packed.x = pack_bf16x2(lo.x, lo.y);
        packed.y = pack_bf16x2(lo.z, lo.w);
        packed.z = pack_bf16x2(hi.x, hi.y);
        packed.w = pack_bf16x2(hi.z, hi.w);
        *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(out) + (size_t)t * H + h) = packed;
    } else {
        float* o = static_cast<float*>(out) + (size_t)t * H + h;
        *reinterpret_cast<f32x4*>(o) = lo;
        *reinterpret_cast<f32x4*>(o + 4) = hi;
    }
}

__global__ void k_stage_accumulate(int E, const int32_t* __restrict__ counts, int64_t* __restrict__ log) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e < E) log[e] += counts[e];
}

template <bool kOutBf16>
hipError_t launch_combine_ks(dim3 grid, const Shape& s, const int32_t* topk_idx, const float* topk_w,
                             const int32_t* inv_perm, const int32_t* expert_slot, const void* y, bool y_bf16, int ks,
                             long long stride, const float* y_off, const int32_t* n_res, void* out, hipStream_t st) {
#define SAEM_COMBINE(KS)                                                                                            \
    hipLaunchKernelGGL((k_combine<kOutBf16, KS>), grid, dim3(256), 0, st, s.T, s.H, s.E, s.k, s.S, s.slots,      \
                       topk_idx, topk_w, inv_perm, expert_slot, static_cast<const float*>(y), ks, stride, y_off,   \
                       n_res, out)
    if (y_bf16 && y_off)
        hipLaunchKernelGGL((k_combine_y16<kOutBf16, true>), dim3(s.T, (s.H + 2047) / 2048), dim3(256), 0, st, s.T,
                           s.H, s.E, s.k, s.S, s.slots, topk_idx, topk_w, inv_perm, expert_slot,
                           static_cast<const uint16_t*>(y), y_off, n_res, out);
    else if (y_bf16)  // no offloaded outputs given: a copy without their registers (higher occupancy)
        hipLaunchKernelGGL((k_combine_y16<kOutBf16, false>), dim3(s.T, (s.H + 2047) / 2048), dim3(256), 0, st, s.T,
                           s.H, s.E, s.k, s.S, s.slots, topk_idx, topk_w, inv_perm, expert_slot,
                           static_cast<const uint16_t*>(y), y_off, n_res, out);
    else if (ks <= 1) SAEM_COMBINE(1);
    else if (ks <= 2) SAEM_COMBINE(2);
    else SAEM_COMBINE(16);
#undef SAEM_COMBINE
    return hipGetLastError();
}

}  // namespace

hipError_t launch_combine(const Shape& s, const int32_t* topk_idx, const float* topk_w, const int32_t* inv_perm,
                          const int32_t* expert_slot, const void* y, bool y_bf16, int ks, long long y_ks_stride,
                          const float* y_off, const int32_t* n_res, void* out, bool out_bf16, hipStream_t st) {
    if (s.T == 0) return hipSuccess;
    if (ks < 1 || ks > 16 || s.k > 8 || s.S > 8 || (y_bf16 && ks != 1)) return hipErrorInvalidValue;
    const dim3 grid(s.T, (s.H + 1023) / 1024);
    return out_bf16 ? launch_combine_ks<true>(grid, s, topk_idx, topk_w, inv_perm, expert_slot, y, y_bf16, ks,
                                              y_ks_stride, y_off, n_res, out, st)
                    : launch_combine_ks<false>(grid, s, topk_idx, topk_w, inv_perm, expert_slot, y, y_bf16, ks,
                                               y_ks_stride, y_off, n_res, out, st);
}

hipError_t launch_stage_accumulate(int E, const int32_t* counts, int64_t* log, hipStream_t st) {
    if (E == 0) return hipSuccess;
    hipLaunchKernelGGL(k_stage_accumulate, dim3((E + 255) / 256), dim3(256), 0, st, E, counts, log);
    return hipGetLastError();
}

}  // namespace saem
