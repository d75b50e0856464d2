// Device helpers shared by the retrieval and graph-search kernels:
// 16-byte dot products and 64-bit wave exchanges.
#pragma once

#include "common.hpp"

namespace is {

// ---- 16-byte dot products (one 128-bit load of each operand) -------------

struct F32Tag {};
struct BF16Tag {};

__device__ __forceinline__ float dot16(uint4 a, uint4 b, F32Tag) {
    float s = __uint_as_float(a.x) * __uint_as_float(b.x);
    s = fmaf(__uint_as_float(a.y), __uint_as_float(b.y), s);
    s = fmaf(__uint_as_float(a.z), __uint_as_float(b.z), s);
    s = fmaf(__uint_as_float(a.w), __uint_as_float(b.w), s);
    return s;
}

__device__ __forceinline__ float dot16(uint4 a, uint4 b, BF16Tag) {
    // bf16 x bf16 products are exact in fp32
    float s = bf16_lo(a.x) * bf16_lo(b.x);
    s = fmaf(bf16_hi(a.x), bf16_hi(b.x), s);
    s = fmaf(bf16_lo(a.y), bf16_lo(b.y), s);
    s = fmaf(bf16_hi(a.y), bf16_hi(b.y), s);
    s = fmaf(bf16_lo(a.z), bf16_lo(b.z), s);
    s = fmaf(bf16_hi(a.z), bf16_hi(b.z), s);
    s = fmaf(bf16_lo(a.w), bf16_lo(b.w), s);
    s = fmaf(bf16_hi(a.w), bf16_hi(b.w), s);
    return s;
}

// ---- wave helpers ----------------------------------------------------------

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int off) {
    const uint32_t lo = __shfl_xor((uint32_t)v, off, kWave);
    const uint32_t hi = __shfl_xor((uint32_t)(v >> 32), off, kWave);
    return ((uint64_t)hi << 32) | lo;
}

// Lanes below this one whose bit is set in a wave-wide mask.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

}  // namespace is
