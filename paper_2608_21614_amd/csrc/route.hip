// route.hip -- router scores and top-k gate (SAEM Section II-A: top-k gating by a router).
//
// One workgroup owns 16 tokens.  For bf16 the scores come from MFMA
// (v_mfma_f32_16x16x32_bf16): router rows are the M side, the 16 tokens the N
// side, and the 4 waves split H; their partial tiles are added into LDS in
// wave order, so the fp32 scores do not depend on timing.  The top-k then runs
// one wave per token: each lane holds experts lane, lane+64, lane+128,
// lane+192, and k rounds of a wave-wide argmax over (score desc, expert asc)
// select the experts.
#include "common.hpp"
#include "kernels.hpp"

#include <math.h>

namespace saem {
namespace {

constexpr int kTok = 16;         // tokens per workgroup
constexpr int kMtBatch = 4;      // expert tiles of 16 accumulated per pass
constexpr int kLgPitch = 257;    // LDS row pitch of the score tile (E <= 256)

// Top-k of one token's scores held as v[i] = score of expert lane + 64 i.
// Selection order: higher score first, equal scores -> lower expert id.
__device__ void topk_wave(const float (&v)[4], int E, int k, int32_t* out_idx, float* out_w) {
    const int lane = lane_id();
    bool taken[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) taken[i] = (lane + 64 * i) >= E;
    float selv[8];
    int sele[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (j >= k) break;
        float bv = -INFINITY;
        int be = 0x7fffffff;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane + 64 * i;
            if (!taken[i] && (v[i] > bv || (v[i] == bv && e < be))) {
                bv = v[i];
                be = e;
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const float ov = __shfl_xor(bv, off, 64);
            const int oe = __shfl_xor(be, off, 64);
            if (ov > bv || (ov == bv && oe < be)) {
                bv = ov;
                be = oe;
            }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (be == lane + 64 * i) taken[i] = true;
        selv[j] = bv;
        sele[j] = be;
    }
    const float top = selv[0];
    float sum = 0.f, mine = 0.f;
    int mye = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (j >= k) break;
        const float term = (selv[j] == top) ? 1.0f : expf(selv[j] - top);
        sum += term;
        if (j == lane) {
            mine = term;
            mye = sele[j];
        }
    }
    if (lane < k) {
        out_idx[lane] = mye;
        out_w[lane] = mine / sum;
    }
}

// Scores of tokens [t0, t0+16) for all experts into s_lg (bf16 inputs, MFMA).
__device__ void scores_bf16(int T, int H, int E, const uint16_t* __restrict__ x, const uint16_t* __restrict__ wr,
                            int t0, float (*s_lg)[kLgPitch]) {
    const int wave = threadIdx.x >> 6, lane = lane_id();
    const int r = lane & 15, kq = (lane >> 4) * 8;
    const int nsteps = H / 32;
    const int s0 = wave * nsteps / 4, s1 = (wave + 1) * nsteps / 4;
    const int tok = t0 + r;
    const uint16_t* xp = (tok < T) ? x + (size_t)tok * H + kq : nullptr;
    const int n_mt = (E + 15) / 16;
    for (int mt0 = 0; mt0 < n_mt; mt0 += kMtBatch) {
        f32x4 acc[kMtBatch];
        const uint16_t* wp[kMtBatch];
#pragma unroll
        for (int m = 0; m < kMtBatch; ++m) {
            acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int e = (mt0 + m) * 16 + r;
            wp[m] = (mt0 + m < n_mt && e < E) ? wr + (size_t)e * H + kq : nullptr;
        }
        for (int s = s0; s < s1; ++s) {
            const bf16x8 b = xp ? load_bf16x8(xp + s * 32) : zero_bf16x8();
#pragma unroll
            for (int m = 0; m < kMtBatch; ++m) {
                const bf16x8 a = wp[m] ? load_bf16x8(wp[m] + s * 32) : zero_bf16x8();
                acc[m] = mfma16x16x32(a, b, acc[m]);
            }
        }
        // add the waves' partial tiles in a fixed order
        for (int ww = 0; ww < 4; ++ww) {
            if (wave == ww) {
#pragma unroll
                for (int m = 0; m < kMtBatch; ++m) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int e = (mt0 + m) * 16 + (lane >> 4) * 4 + i;
                        if (mt0 + m < n_mt && e < E) s_lg[r][e] += acc[m][i];
                    }
                }
            }
            __syncthreads();
        }
    }
}

// Scores for fp32 inputs: plain fp32 FMA, one (token, expert) dot product per thread pass.
__device__ void scores_f32(int T, int H, int E, const float* __restrict__ x, const float* __restrict__ wr, int t0,
                           float (*s_lg)[kLgPitch]) {
    const int tt = threadIdx.x >> 4, el = threadIdx.x & 15;
    const int t = t0 + tt;
    if (t < T) {
        for (int e = el; e < E; e += 16) {
            float acc = 0.f;
            for (int h = 0; h < H; ++h) acc = fmaf(x[(size_t)t * H + h], wr[(size_t)e * H + h], acc);
            s_lg[tt][e] = acc;
        }
    }
    __syncthreads();
}

template <bool kBf16>
__global__ void __launch_bounds__(256) k_route_topk(int T, int H, int E, int k, const void* __restrict__ x,
                                                    const void* __restrict__ wr, const float* __restrict__ bias,
                                                    float* __restrict__ logits, int logits_in,
                                                    int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    __shared__ float s_lg[kTok][kLgPitch];
    const int t0 = blockIdx.x * kTok;
    const int wave = threadIdx.x >> 6, lane = lane_id();
    if (!logits_in) {
        for (int i = threadIdx.x; i < kTok * kLgPitch; i += blockDim.x) (&s_lg[0][0])[i] = 0.f;
        __syncthreads();
        if (kBf16)
            scores_bf16(T, H, E, static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(wr), t0, s_lg);
        else
            scores_f32(T, H, E, static_cast<const float*>(x), static_cast<const float*>(wr), t0, s_lg);
    }
    for (int tt = wave; tt < kTok; tt += 4) {
        const int t = t0 + tt;
        if (t >= T) break;
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = lane + 64 * i;
            v[i] = -INFINITY;
            if (e < E) {
                if (logits_in) {
                    v[i] = logits[(size_t)t * E + e];
                } else {
                    v[i] = s_lg[tt][e] + (bias ? bias[e] : 0.f);
                    logits[(size_t)t * E + e] = v[i];
                }
            }
        }
        topk_wave(v, E, k, topk_idx + (size_t)t * k, topk_w + (size_t)t * k);
    }
}

}  // namespace

hipError_t launch_route_topk(const Shape& s, const void* x, const void* w_router, const float* bias, float* logits,
                             bool logits_in, int32_t* topk_idx, float* topk_w, hipStream_t st) {
    if (s.T == 0) return hipSuccess;
    dim3 grid((s.T + kTok - 1) / kTok), block(256);
    if (s.bf16)
        hipLaunchKernelGGL(k_route_topk<true>, grid, block, 0, st, s.T, s.H, s.E, s.k, x, w_router, bias, logits,
                           logits_in ? 1 : 0, topk_idx, topk_w);
    else
        hipLaunchKernelGGL(k_route_topk<false>, grid, block, 0, st, s.T, s.H, s.E, s.k, x, w_router, bias, logits,
                           logits_in ? 1 : 0, topk_idx, topk_w);
    return hipGetLastError();
}

}  // namespace saem
