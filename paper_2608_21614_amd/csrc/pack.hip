// pack.hip -- expert weights into the MFMA tile layout.
//
// A K-contiguous matrix W[R][K] (R % 16 == 0, K % 32 == 0) is stored as blocks
// of 16 rows x 32 columns; block (rt, s) covers rows 16*rt .. 16*rt+15 and
// columns 32*s .. 32*s+31 and sits at element offset (rt * K/32 + s) * 512.
// Inside a block, element 8*l + i holds W[16*rt + l%16][32*s + 8*(l/16) + i]:
// lane l of a wave reads its MFMA A operand (row l%16, 8 consecutive K values)
// as one 16-byte load, and a wave reads a whole block as 1 KB of contiguous
// memory.  Expert weights are packed once, when they are loaded into a slot
// (the fixed per-layer expert slots of SAEM Section IV-C.1); every forward then
// streams them with fully contiguous wave loads.
#include "common.hpp"
#include "kernels.hpp"

namespace saem {
namespace {

// One thread moves 8 consecutive K elements of one row (elt = 2 or 4 bytes).
template <typename T>
__global__ void __launch_bounds__(256)
    k_pack(const T* __restrict__ src, T* __restrict__ dst, long long rows, long long K) {
    const long long nsteps = K / 32;
    const long long chunks = rows * (K / 8);  // 8-element chunks
    for (long long c = (long long)blockIdx.x * 256 + threadIdx.x; c < chunks; c += (long long)gridDim.x * 256) {
        const long long blk = c / 64, l = c % 64;
        const long long rt = blk / nsteps, s = blk % nsteps;
        const long long row = 16 * rt + (l & 15), col = 32 * s + 8 * (l >> 4);
        const T* in = src + row * K + col;
        T* out = dst + blk * 512 + l * 8;
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = in[i];
    }
}

}  // namespace

hipError_t launch_pack_weights(const void* src, void* dst, long long rows, long long K, bool bf16, hipStream_t st) {
    const long long chunks = rows * (K / 8);
    if (chunks == 0) return hipSuccess;
    long long grid = (chunks + 255) / 256;
    if (grid > 65536) grid = 65536;
    if (bf16)
        hipLaunchKernelGGL(k_pack<uint16_t>, dim3((unsigned)grid), dim3(256), 0, st, static_cast<const uint16_t*>(src),
                           static_cast<uint16_t*>(dst), rows, K);
    else
        hipLaunchKernelGGL(k_pack<float>, dim3((unsigned)grid), dim3(256), 0, st, static_cast<const float*>(src),
                           static_cast<float*>(dst), rows, K);
    return hipGetLastError();
}

}  // namespace saem
