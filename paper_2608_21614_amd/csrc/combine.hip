// combine.hip -- merge of the expert outputs back to token order
// (SAEM Section IV-D.2).  A gather in a fixed order, with no atomics, so two
// runs give bitwise-identical outputs; the paper's atomic accumulation is not
// reproducible (Section V-C).
//
// Workgroup = one token x 1024 hidden columns (4 per thread, 16-byte loads):
//   acc = 0
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

template <bool kOutBf16>
__global__ void __launch_bounds__(256)
    k_combine(int T, int H, int E, int k, int S, int slots, const int32_t* __restrict__ topk_idx,
              const float* __restrict__ topk_w, const int32_t* __restrict__ inv_perm,
              const int32_t* __restrict__ expert_slot, const float* __restrict__ y, int ks, long long stride,
              const float* __restrict__ y_off, const int32_t* __restrict__ n_res_p, void* __restrict__ out) {
    const int t = blockIdx.x;
    const int h = (blockIdx.y * 256 + threadIdx.x) * 4;
    if (h >= H) return;
    const int P = T * k;
    const int nres = y_off ? *n_res_p : 0;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
        const int q = t * k + j;
        const int e = topk_idx[q];
        if (e < 0 || e >= E) continue;
        const int p = inv_perm[q];
        if (p < 0 || p >= P) continue;
        const float w = topk_w[q];
        if (is_resident(expert_slot[e], slots)) {
            acc += w * sum_chunks(y, ks, stride, (size_t)p * H + h);
        } else if (y_off && p >= nres) {
            acc += w * *reinterpret_cast<const f32x4*>(y_off + (size_t)(p - nres) * H + h);
        }
    }
    for (int s = 0; s < S; ++s) {
        const size_t row = (size_t)P + (size_t)s * T + t;
        acc += sum_chunks(y, ks, stride, row * H + h);
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

__global__ void k_stage_accumulate(int E, const int32_t* __restrict__ counts, int64_t* __restrict__ log) {
    const int e = blockIdx.x * blockDim.x + threadIdx.x;
    if (e < E) log[e] += counts[e];
}

}  // namespace

hipError_t launch_combine(const Shape& s, const int32_t* topk_idx, const float* topk_w, const int32_t* inv_perm,
                          const int32_t* expert_slot, const float* y, int ks, long long y_ks_stride,
                          const float* y_off, const int32_t* n_res, void* out, bool out_bf16, hipStream_t st) {
    if (s.T == 0) return hipSuccess;
    dim3 grid(s.T, (s.H + 1023) / 1024), block(256);
    if (out_bf16)
        hipLaunchKernelGGL(k_combine<true>, grid, block, 0, st, s.T, s.H, s.E, s.k, s.S, s.slots, topk_idx, topk_w,
                           inv_perm, expert_slot, y, ks, y_ks_stride, y_off, n_res, out);
    else
        hipLaunchKernelGGL(k_combine<false>, grid, block, 0, st, s.T, s.H, s.E, s.k, s.S, s.slots, topk_idx, topk_w,
                           inv_perm, expert_slot, y, ks, y_ks_stride, y_off, n_res, out);
    return hipGetLastError();
}

hipError_t launch_stage_accumulate(int E, const int32_t* counts, int64_t* log, hipStream_t st) {
    if (E == 0) return hipSuccess;
    hipLaunchKernelGGL(k_stage_accumulate, dim3((E + 255) / 256), dim3(256), 0, st, E, counts, log);
    return hipGetLastError();
}

}  // namespace saem
