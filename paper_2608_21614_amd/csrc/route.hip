// route.hip -- router scores and top-k gate (SAEM Section II-A: top-k gating by
// a router), and the decode front end (scores + top-k + repacking).
//
// Scores run on MFMA (v_mfma_f32_16x16x32_bf16, or v_mfma_f32_16x16x4_f32 for
// fp32 inputs): router rows are the M side, 16 tokens the N side.
//
//  * T > 64 (prefill): k_route_topk, 8 tokens per 1024-thread workgroup whose
//    16 waves split K and add their partial tiles in a fixed order.
// The top-k takes one wave per token (topk_block: k rounds of a wave argmax).
//  * T <= 64 (decode): k_router_partial spreads the scores over one workgroup
//    per K slice (a single CU cannot stream the batch and the router fast
//    enough), then k_route_finish adds each token's slices in order and runs its
//    top-k, one wave per token over many CUs.  The fused forward and
//    moe_route_topk use the same two kernels, so both give bit-identical scores;
//    the repacking follows in k_repack.
#include "block_ops.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

// Tokens per workgroup: 8 of the 16-token MFMA tile, so that a 2048-token batch fills all
// 256 CUs (every workgroup streams the whole router matrix, whatever its token count).
constexpr int kRouteRows = 8;

template <bool kBf16>
__global__ void __launch_bounds__(kFrontThreads)
    k_route_topk(int T, int H, int E, int k, const void* __restrict__ x, const void* __restrict__ wr,
                 const float* __restrict__ bias, float* __restrict__ logits, int logits_in,
                 int32_t* __restrict__ topk_idx, float* __restrict__ topk_w) {
    __shared__ float s_lg[16 * kLgPitch];
    __shared__ float s_red[kFrontWaves * 16 * kScoreChunk];
    __shared__ float s_selv[64 * 8];
    __shared__ int s_sele[64 * 8];
    const int t0 = blockIdx.x * kRouteRows;
    const int tend = min(T, t0 + kRouteRows);  // the MFMA tile's rows past it stay zero
    if (!logits_in) {
        if (kBf16)
            router_scores_mfma<uint16_t, 1, kFrontWaves>(tend, H, E, static_cast<const uint16_t*>(x),
                                                         static_cast<const uint16_t*>(wr), bias, t0, s_lg, s_red);
        else
            router_scores_mfma<float, 1, kFrontWaves>(tend, H, E, static_cast<const float*>(x),
                                                      static_cast<const float*>(wr), bias, t0, s_lg, s_red);
    }
    const int rows = tend - t0;
    // scores <-> global, coalesced
    for (int idx = threadIdx.x; idx < rows * E; idx += kFrontThreads) {
        const int row = idx / E, e = idx % E;
        if (logits_in) s_lg[row * kLgPitch + e] = logits[(size_t)(t0 + row) * E + e];
        else logits[(size_t)(t0 + row) * E + e] = s_lg[row * kLgPitch + e];
    }
    __syncthreads();
    topk_block(s_lg, rows, E, k, t0, topk_idx, topk_w, nullptr, s_selv, s_sele);
}

// Decode batches: part[slice][t][e] = sum over the slice's K steps of x[t] . w_router[e].
// One workgroup per (K slice, chunk of 64 experts); wave w covers tokens
// 16w .. 16w+15; MFMA on bf16 (16x16x32) or fp32 (16x16x4) operands.
template <typename Elt>
__global__ void __launch_bounds__(256)
    k_router_partial(int T, int H, int E, const void* __restrict__ x, const void* __restrict__ wr, int nsl,
                     float* __restrict__ part) {
    const int slice = blockIdx.x;
    const int nst = H / 32, s0 = slice * nst / nsl, s1 = (slice + 1) * nst / nsl;
    float* out = part + (size_t)slice * 64 * E;
    const int wave = threadIdx.x >> 6, lane = lane_id();
    const int r = lane & 15, kq = (lane >> 4) * 8;
    if (16 * wave >= T) return;
    const int tok = 16 * wave + r;
    const Elt* xp = (tok < T) ? static_cast<const Elt*>(x) + (size_t)tok * H + kq : nullptr;
    {
        const int c0 = blockIdx.y * kScoreChunk;
        f32x4 acc[4];
        const Elt* wp[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            acc[m] = f32x4{0.f, 0.f, 0.f, 0.f};
            const int e = c0 + 16 * m + r;
            wp[m] = (e < E) ? static_cast<const Elt*>(wr) + (size_t)e * H + kq : nullptr;
        }
        for (int s = s0; s < s1; s += 4) {
            Frag8<Elt> A[4][4], B[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const bool ok = s + u < s1;
                B[u] = (ok && xp) ? load_frag(xp + (s + u) * 32) : zero_frag<Elt>();
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    A[u][m] = (ok && wp[m]) ? load_frag(wp[m] + (s + u) * 32) : zero_frag<Elt>();
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int m = 0; m < 4; ++m)
                    if (c0 + 16 * m < E) acc[m] = mma_frag(A[u][m], B[u], acc[m]);
        }
        if (tok < T) {
#pragma unroll
            for (int m = 0; m < 4; ++m)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int e = c0 + 16 * m + 4 * (lane >> 4) + i;
                    if (e < E) out[tok * E + e] = acc[m][i];
                }
        }
    }
}

// Decode front end, second step: one wave per token adds the token's K-sliced
// partial scores in slice order (+ bias) and writes them to logits (or reads the
// caller's scores), then picks the token's top-k in rank order with k rounds of
// a wave argmax over integer keys with the scores' order: lane l holds experts
// l, l + 64, l + 128, l + 192, offers its best open one (largest key, then lowest
// id), and the wave takes the largest key and, among the lanes offering it, the
// lowest id.  The gate of choice j is exp(s_j - s_0) / sum_j' exp(s_j' - s_0),
// summed in j order; a score equal to the top one contributes exactly 1.
// NS: expert slots per lane (E <= 64 NS).
template <int NS>
__global__ void __launch_bounds__(256)
    k_route_finish(int T, int E, int k, const float* __restrict__ part, int nsl, const float* __restrict__ bias,
                   float* __restrict__ logits, int logits_in, int32_t* __restrict__ topk_idx,
                   float* __restrict__ topk_w) {
    const int lane = lane_id();
    const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (t >= T) return;  // the whole wave
    float v[NS];
    int key[NS];
    bool open[NS];
#pragma unroll
    for (int sl = 0; sl < NS; ++sl) {
        open[sl] = lane + kWave * sl < E;
        v[sl] = 0.f;
    }
    if (logits_in) {
#pragma unroll
        for (int sl = 0; sl < NS; ++sl)
            if (open[sl]) v[sl] = logits[(size_t)t * E + lane + kWave * sl];
    } else {
        // all slots' loads of a batch of 16 slices in flight together, bias included
        float bv[NS];
#pragma unroll
        for (int sl = 0; sl < NS; ++sl) bv[sl] = (open[sl] && bias) ? bias[lane + kWave * sl] : 0.f;
        for (int b = 0; b < nsl; b += 16) {
            float q[NS][16];
#pragma unroll
            for (int sl = 0; sl < NS; ++sl) {
                const float* p = part + (size_t)t * E + (open[sl] ? lane + kWave * sl : 0);
#pragma unroll
                for (int j = 0; j < 16; ++j) q[sl][j] = (b + j < nsl) ? p[(size_t)(b + j) * 64 * E] : 0.f;
            }
#pragma unroll
            for (int sl = 0; sl < NS; ++sl)
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    if (b + j < nsl) v[sl] = (b + j == 0) ? q[sl][j] : v[sl] + q[sl][j];
        }
#pragma unroll
        for (int sl = 0; sl < NS; ++sl)
            if (open[sl]) {
                v[sl] += bv[sl];
                logits[(size_t)t * E + lane + kWave * sl] = v[sl];
            }
    }
#pragma unroll
    for (int sl = 0; sl < NS; ++sl) key[sl] = score_key(v[sl]);
    float selv[8];
    int sele[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        selv[j] = 0.f;
        sele[j] = -1;
        if (j >= k) continue;  // uniform
        int kb = INT_MIN, eb = INT_MAX;
#pragma unroll
        for (int sl = 0; sl < NS; ++sl)
            if (open[sl] && (eb == INT_MAX || key[sl] > kb)) {
                kb = key[sl];
                eb = lane + kWave * sl;
            }
        const int m = wave_max_i32(eb != INT_MAX ? kb : INT_MIN);
        const int e = wave_min_i32((eb != INT_MAX && kb == m) ? eb : INT_MAX);  // never INT_MAX: k <= E
#pragma unroll
        for (int sl = 0; sl < NS; ++sl)
            if (lane + kWave * sl == e) open[sl] = false;
        const int es = e >> 6, el = e & 63;
        float ve = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[0]), el));
#pragma unroll
        for (int sl = 1; sl < NS; ++sl)
            if (es == sl) ve = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v[sl]), el));
        selv[j] = ve;
        sele[j] = e;
    }
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (j < k) sum += (selv[j] == selv[0]) ? 1.0f : expf(selv[j] - selv[0]);
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (j < k && lane == j) {
            const float term = (selv[j] == selv[0]) ? 1.0f : expf(selv[j] - selv[0]);
            topk_idx[(size_t)t * k + j] = sele[j];
            topk_w[(size_t)t * k + j] = term / sum;
        }
}

hipError_t launch_small(const Shape& s, const void* x, const void* w_router, const float* bias, float* logits,
                        bool logits_in, int32_t* topk_idx, float* topk_w, float* part, hipStream_t st) {
    const int nsl = router_slices(s);
    if (!logits_in && s.T > 0) {
        if (s.bf16)
            hipLaunchKernelGGL(k_router_partial<uint16_t>, dim3(nsl, (s.E + kScoreChunk - 1) / kScoreChunk), dim3(256),
                               0, st, s.T, s.H, s.E, x, w_router, nsl, part);
        else
            hipLaunchKernelGGL(k_router_partial<float>, dim3(nsl, (s.E + kScoreChunk - 1) / kScoreChunk), dim3(256), 0,
                               st, s.T, s.H, s.E, x, w_router, nsl, part);
    }
    const dim3 grid((s.T + 3) / 4);
    const int li = logits_in ? 1 : 0;
    if (s.E <= 64)
        hipLaunchKernelGGL(k_route_finish<1>, grid, dim3(256), 0, st, s.T, s.E, s.k, part, nsl, bias, logits, li,
                           topk_idx, topk_w);
    else if (s.E <= 128)
        hipLaunchKernelGGL(k_route_finish<2>, grid, dim3(256), 0, st, s.T, s.E, s.k, part, nsl, bias, logits, li,
                           topk_idx, topk_w);
    else
        hipLaunchKernelGGL(k_route_finish<4>, grid, dim3(256), 0, st, s.T, s.E, s.k, part, nsl, bias, logits, li,
                           topk_idx, topk_w);
    return hipGetLastError();
}

}  // namespace

bool front_small_fits(const Shape& s) { return s.T <= 64; }

int router_slices(const Shape& s) {
    if (!front_small_fits(s)) return 0;
    const int n = (s.H / 32) / 4;  // about 4 K steps of 32 per workgroup
    return n < 1 ? 1 : (n > 64 ? 64 : n);
}

hipError_t launch_route_topk(const Shape& s, const void* x, const void* w_router, const float* bias, float* logits,
                             bool logits_in, int32_t* topk_idx, float* topk_w, float* part, hipStream_t st) {
    if (s.T == 0) return hipSuccess;
    if (front_small_fits(s)) return launch_small(s, x, w_router, bias, logits, logits_in, topk_idx, topk_w, part, st);
    const int li = logits_in ? 1 : 0;
    dim3 grid((s.T + kRouteRows - 1) / kRouteRows), block(kFrontThreads);
    if (s.bf16)
        hipLaunchKernelGGL(k_route_topk<true>, grid, block, 0, st, s.T, s.H, s.E, s.k, x, w_router, bias, logits, li,
                           topk_idx, topk_w);
    else
        hipLaunchKernelGGL(k_route_topk<false>, grid, block, 0, st, s.T, s.H, s.E, s.k, x, w_router, bias, logits,
                           li, topk_idx, topk_w);
    return hipGetLastError();
}

}  // namespace saem
