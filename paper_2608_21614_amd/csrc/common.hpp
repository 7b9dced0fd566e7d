// common.hpp -- device helpers shared by the gfx950 kernels of libsaem_moe.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace saem {

// bf16 data are carried as raw 16-bit patterns; MFMA operands are 8 x bf16 per lane.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

// 16-byte global load of 8 bf16 as an MFMA operand.
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// Streaming (read-once) variant: the weights of an expert are read once per call.
__device__ __forceinline__ bf16x8 load_bf16x8_stream(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}

__device__ __forceinline__ bf16x8 zero_bf16x8() { return __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u}); }

// D(16x16 fp32) += A(16x32 bf16) * B(32x16 bf16).
// Lane l supplies A row (l % 16) and B column (l % 16), each with the 8
// consecutive K values 8*(l/16) .. 8*(l/16)+7; it receives D rows
// 4*(l/16) .. 4*(l/16)+3 of column (l % 16).
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// MFMA operand fragment: 8 consecutive K values of one lane (its row, or its
// column, and K offset 8*(lane/16) inside a 32-wide K step).  bf16 feeds one
// 16x16x32 MFMA; fp32 feeds eight 16x16x4 MFMAs, MFMA i taking value i of every
// lane, i.e. K indices {i, 8+i, 16+i, 24+i} of the step.  Both operands use the
// same assignment, so every product of the step is summed exactly once.
template <typename Elt>
struct Frag8;
template <>
struct Frag8<uint16_t> {
    bf16x8 v;
};
template <>
struct Frag8<float> {
    f32x4 lo, hi;
};

__device__ __forceinline__ Frag8<uint16_t> load_frag(const uint16_t* p) { return {load_bf16x8(p)}; }
__device__ __forceinline__ Frag8<float> load_frag(const float* p) {
    const f32x4* q = reinterpret_cast<const f32x4*>(p);
    return {q[0], q[1]};
}
// Read-once operands (an expert's weights at decode): non-temporal loads.
__device__ __forceinline__ Frag8<uint16_t> load_frag_stream(const uint16_t* p) { return {load_bf16x8_stream(p)}; }
__device__ __forceinline__ Frag8<float> load_frag_stream(const float* p) {
    const f32x4* q = reinterpret_cast<const f32x4*>(p);
    return {__builtin_nontemporal_load(q), __builtin_nontemporal_load(q + 1)};
}
template <typename Elt>
__device__ __forceinline__ Frag8<Elt> zero_frag();
template <>
__device__ __forceinline__ Frag8<uint16_t> zero_frag<uint16_t>() { return {zero_bf16x8()}; }
template <>
__device__ __forceinline__ Frag8<float> zero_frag<float>() {
    return {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
}

__device__ __forceinline__ f32x4 mma_frag(const Frag8<uint16_t>& a, const Frag8<uint16_t>& b, f32x4 c) {
    return mfma16x16x32(a.v, b.v, c);
}
__device__ __forceinline__ f32x4 mma_frag(const Frag8<float>& a, const Frag8<float>& b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.x, b.lo.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.y, b.lo.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.z, b.lo.z, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.lo.w, b.lo.w, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.x, b.hi.x, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.y, b.hi.y, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.z, b.hi.z, c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.hi.w, b.hi.w, c, 0, 0, 0);
    return c;
}

// silu(z) = z / (1 + e^-z), with the hardware reciprocal (about 1 ulp) instead of a
// correctly rounded divide; z = -inf gives NaN, as the quotient does.
__device__ __forceinline__ float silu(float z) { return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z)); }

// Four bf16 values (8 bytes) widened to fp32.
__device__ __forceinline__ f32x4 bf16x4_to_f32(u32x2 v) {
    return f32x4{__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u), __uint_as_float(v.y << 16),
                 __uint_as_float(v.y & 0xffff0000u)};
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Residency rule of the ABI: resident iff 0 <= slot < slots.
__device__ __forceinline__ bool is_resident(int32_t slot, int slots) { return slot >= 0 && slot < slots; }

}  // namespace saem
