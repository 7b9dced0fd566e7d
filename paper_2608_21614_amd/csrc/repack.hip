// repack.hip -- expert-aligned token repacking with the residency split
// (SAEM Section IV-E.1; partition by residency map, Section IV-D.2).
//
// One workgroup of 1024 threads does the whole batch (T*k pairs is at most a
// few tens of thousands):
//   1. histogram of the pairs per expert with LDS atomics (order-free);
//   2. one wave scans the counts in group order -- resident experts by id,
//      then offloaded experts by id -- into segment starts and n_res;
//   3. the pairs are scattered in chunks of 1024, one per thread.  Inside a
//      wave, lanes holding the same expert are found with 8 ballots over the
//      bits of the expert id, and a lane's rank is the popcount of the matching
//      lanes below it; per-wave counts go to LDS so each wave adds the counts of
//      the waves before it.  Pairs keep their index order inside an expert:
//      a stable counting sort, with no global atomics.
// A second small kernel packs the offloaded rows for the host.
#include "common.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

constexpr int kRepackThreads = 1024;
constexpr int kRepackWaves = kRepackThreads / kWave;

__global__ void __launch_bounds__(kRepackThreads)
    k_repack(int T, int E, int k, int slots, const int32_t* __restrict__ topk_idx,
             const int32_t* __restrict__ expert_slot, int32_t* __restrict__ counts, int32_t* __restrict__ seg_start,
             int32_t* __restrict__ perm, int32_t* __restrict__ inv_perm, int32_t* __restrict__ n_res) {
    __shared__ int s_cnt[256];
    __shared__ int s_base[256];
    __shared__ int s_res[256];
    __shared__ int s_wcnt[kRepackWaves][256];
    __shared__ int s_nres;
    const int tid = threadIdx.x, wave = tid >> 6, lane = lane_id();
    const int P = T * k;

    for (int e = tid; e < 256; e += kRepackThreads) {
        s_cnt[e] = 0;
        s_res[e] = (e < E) ? (is_resident(expert_slot[e], slots) ? 1 : 0) : 0;
    }
    __syncthreads();
    for (int q = tid; q < P; q += kRepackThreads) {
        const int e = topk_idx[q];
        if (e >= 0 && e < E) atomicAdd(&s_cnt[e], 1);
    }
    __syncthreads();

    if (wave == 0) {
        // lane owns experts 4*lane .. 4*lane+3
        int rs = 0, os = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 4 * lane + i;
            if (e < E) {
                if (s_res[e]) rs += s_cnt[e];
                else os += s_cnt[e];
            }
        }
        int rinc = rs, oinc = os;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int a = __shfl_up(rinc, off, 64);
            const int b = __shfl_up(oinc, off, 64);
            if (lane >= off) {
                rinc += a;
                oinc += b;
            }
        }
        const int rtot = __shfl(rinc, 63, 64);
        int rp = rinc - rs, op = rtot + (oinc - os);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = 4 * lane + i;
            if (e < E) {
                if (s_res[e]) {
                    s_base[e] = rp;
                    rp += s_cnt[e];
                } else {
                    s_base[e] = op;
                    op += s_cnt[e];
                }
            }
        }
        if (lane == 0) s_nres = rtot;
    }
    __syncthreads();
    for (int e = tid; e < E; e += kRepackThreads) {
        counts[e] = s_cnt[e];
        seg_start[e] = s_base[e];
    }
    if (tid == 0) *n_res = s_nres;

    const unsigned long long lt_mask = (1ull << lane) - 1ull;
    for (int c0 = 0; c0 < P; c0 += kRepackThreads) {
        for (int i = tid; i < kRepackWaves * 256; i += kRepackThreads) (&s_wcnt[0][0])[i] = 0;
        __syncthreads();
        const int q = c0 + tid;
        const int e = (q < P) ? topk_idx[q] : -1;
        const bool valid = (e >= 0 && e < E);
        unsigned long long m = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = valid && ((e >> b) & 1);
            const unsigned long long bb = __ballot(bit);
            m &= bit ? bb : ~bb;
        }
        const int rank = __popcll(m & lt_mask);
        if (valid && rank == 0) s_wcnt[wave][e] = __popcll(m);
        __syncthreads();
        if (valid) {
            int p = s_base[e] + rank;
            for (int w = 0; w < wave; ++w) p += s_wcnt[w][e];
            perm[p] = q;
            inv_perm[q] = p;
        } else if (q < P) {
            inv_perm[q] = -1;
        }
        __syncthreads();
        for (int ee = tid; ee < E; ee += kRepackThreads) {
            int sum = 0;
#pragma unroll
            for (int w = 0; w < kRepackWaves; ++w) sum += s_wcnt[w][ee];
            s_base[ee] += sum;
        }
        __syncthreads();
    }
}

// off_rows[p - n_res] = x[perm[p] / k]; off_w[p - n_res] = topk_w[perm[p]].
__global__ void __launch_bounds__(256)
    k_offload_pack(int T, int k, int row_bytes, const uint8_t* __restrict__ x, const float* __restrict__ topk_w,
                   const int32_t* __restrict__ perm, const int32_t* __restrict__ n_res_p, uint8_t* __restrict__ off_rows,
                   float* __restrict__ off_w) {
    const int P = T * k;
    const int nres = *n_res_p;
    const int chunks = row_bytes / 16;
    for (int p = nres + (int)blockIdx.x; p < P; p += gridDim.x) {
        const int q = perm[p];
        if (q < 0 || q >= P) continue;  // rows of dropped pairs are left as they are
        const int t = q / k;
        if (off_rows) {
            const u32x4* src = reinterpret_cast<const u32x4*>(x + (size_t)t * row_bytes);
            u32x4* dst = reinterpret_cast<u32x4*>(off_rows + (size_t)(p - nres) * row_bytes);
            for (int c = threadIdx.x; c < chunks; c += blockDim.x) dst[c] = src[c];
        }
        if (off_w && threadIdx.x == 0) off_w[p - nres] = topk_w[q];
    }
}

}  // namespace

hipError_t launch_repack(const Shape& s, const int32_t* topk_idx, const int32_t* expert_slot, int32_t* counts,
                         int32_t* seg_start, int32_t* perm, int32_t* inv_perm, int32_t* n_res, hipStream_t st) {
    hipLaunchKernelGGL(k_repack, dim3(1), dim3(kRepackThreads), 0, st, s.T, s.E, s.k, s.slots, topk_idx, expert_slot,
                       counts, seg_start, perm, inv_perm, n_res);
    return hipGetLastError();
}

hipError_t launch_offload_pack(const Shape& s, const void* x, const float* topk_w, const int32_t* perm,
                               const int32_t* n_res, void* off_rows, float* off_w, hipStream_t st) {
    const int P = s.T * s.k;
    if (P == 0 || (!off_rows && !off_w)) return hipSuccess;
    const int row_bytes = s.H * (s.bf16 ? 2 : 4);
    const int grid = P < 1024 ? P : 1024;
    hipLaunchKernelGGL(k_offload_pack, dim3(grid), dim3(256), 0, st, s.T, s.k, row_bytes,
                       static_cast<const uint8_t*>(x), topk_w, perm, n_res, static_cast<uint8_t*>(off_rows), off_w);
    return hipGetLastError();
}

}  // namespace saem
