// Device helpers shared by the gfx950 kernels of libinferscale.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace is {

constexpr int kWave = 64;  // CDNA wavefront width

// ---- bf16 <-> fp32 ---------------------------------------------------------

__device__ __forceinline__ float bf16_lo(uint32_t packed) {
    return __uint_as_float(packed << 16);
}
__device__ __forceinline__ float bf16_hi(uint32_t packed) {
    return __uint_as_float(packed & 0xFFFF0000u);
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values -> packed bf16 (lo in bits 0..15), round to nearest, ties
// to even (one v_cvt_pk_bf16_f32 on gfx950; NaN stays a quiet NaN).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

// Integer minimum of two 64-bit values. (HIP's min() with mixed operand
// types promotes both to double; these keep integer arithmetic.)
__device__ __forceinline__ int64_t min_i64(int64_t a, int64_t b) { return a < b ? a : b; }

// ---- ranking keys ----------------------------------------------------------
// A 64-bit key whose unsigned order is the rank order (score desc, id asc):
// high word = order-preserving image of the fp32 score (-0 folded onto +0,
// NaN mapped below every number), low word = ~id.

__device__ __forceinline__ uint32_t score_order_bits(float s) {
    uint32_t u = __float_as_uint(s);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0u;  // NaN: lowest
    if (u == 0x80000000u) u = 0u;                     // -0 -> +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float score_from_order_bits(uint32_t o) {
    if (o == 0u) return __uint_as_float(0x7FC00000u);
    uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return __uint_as_float(u);
}

__device__ __forceinline__ uint64_t rank_key(float s, uint32_t id) {
    return ((uint64_t)score_order_bits(s) << 32) | (uint64_t)(~id);
}

__device__ __forceinline__ uint32_t key_id(uint64_t key) { return ~(uint32_t)key; }
__device__ __forceinline__ float key_score(uint64_t key) {
    return score_from_order_bits((uint32_t)(key >> 32));
}

// ---- wave reductions ---------------------------------------------------------

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Inclusive prefix sum of a 64-bit value across the lanes of a wave.
__device__ __forceinline__ int64_t wave_incl_scan(int64_t v, int lane) {
#pragma unroll
    for (int off = 1; off < kWave; off <<= 1) {
        const uint32_t lo = __shfl_up((uint32_t)v, off, kWave);
        const int32_t hi = __shfl_up((int32_t)(v >> 32), off, kWave);
        const int64_t o = (int64_t)(((uint64_t)(uint32_t)hi << 32) | lo);
        if (lane >= off) v += o;
    }
    return v;
}

}  // namespace is
