// repack.hip -- expert-aligned token repacking with the residency split
// (SAEM Section IV-E.1; partition by residency map, Section IV-D.2).
//
// A stable counting sort over the T*k pairs (repack_chunks in block_ops.hpp).
// Up to 512 pairs (a decode batch): one workgroup of 256 threads.  Otherwise
// chunks of 1024 pairs, split into contiguous ranges over up to kRepackGroups
// workgroups of 1024 threads; every workgroup counts the whole batch itself, so
// none waits for another, and the result does not depend on the split.  A
// second small kernel packs the offloaded rows for the host when the FFN does
// not (moe_repack on its own, fp32 prefill).
#include "block_ops.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

// Workgroups of one repack: each counts all T*k ids, so more groups cost L2 reads
// (groups x T*k) and fewer cost chunk passes (chunks / groups in sequence).
constexpr int kRepackGroups = 128;

template <int NT>
__global__ void __launch_bounds__(NT)
    k_repack(int T, int E, int k, int slots, int chunks, const int32_t* __restrict__ topk_idx,
             const int32_t* __restrict__ expert_slot, int32_t* __restrict__ counts, int32_t* __restrict__ seg_start,
             int32_t* __restrict__ perm, int32_t* __restrict__ inv_perm, int32_t* __restrict__ n_res) {
    __shared__ int s_lds[repack_lds_ints<NT>()];
    const int g = blockIdx.x, G = gridDim.x;
    const int c_begin = (int)((long long)chunks * g / G), c_end = (int)((long long)chunks * (g + 1) / G);
    repack_chunks<NT>(T, E, k, slots, c_begin, c_end, topk_idx, expert_slot, counts, seg_start, perm, inv_perm, n_res,
                      s_lds);
}

// off_rows[p - n_res] = x[perm[p] / k]; off_w[p - n_res] = topk_w[perm[p]].
__global__ void __launch_bounds__(256)
    k_offload_pack(int T, int k, int row_bytes, const uint8_t* __restrict__ x, const float* __restrict__ topk_w,
                   const int32_t* __restrict__ perm, const int32_t* __restrict__ n_res_p,
                   uint8_t* __restrict__ off_rows,
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
    const int P = s.T * s.k;
    if (P <= 512) {  // a decode batch: one workgroup of 256 threads, up to two chunks
        const int chunks = (P + 255) / 256;
        hipLaunchKernelGGL(k_repack<256>, dim3(1), dim3(256), 0, st, s.T, s.E, s.k, s.slots, chunks, topk_idx,
                           expert_slot, counts, seg_start, perm, inv_perm, n_res);
        return hipGetLastError();
    }
    const int chunks = (P + kFrontThreads - 1) / kFrontThreads;
    const int groups = chunks < kRepackGroups ? chunks : kRepackGroups;
    hipLaunchKernelGGL(k_repack<kFrontThreads>, dim3((unsigned)groups), dim3(kFrontThreads), 0, st, s.T, s.E, s.k,
                       s.slots, chunks, topk_idx, expert_slot, counts, seg_start, perm, inv_perm, n_res);
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
