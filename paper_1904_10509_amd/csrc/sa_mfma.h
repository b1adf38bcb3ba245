// gfx950 matrix-core helpers for the bf16 attention kernels.
//
// One MFMA v_mfma_f32_16x16x32_bf16 computes D[16x16] += A[16x32] * B[32x16]
// across a 64-lane wavefront.  With lane = 16 * g + r (g = lane / 16,
// r = lane % 16):
//   A operand: lane holds A[r][8g .. 8g+7]        (8 bf16)
//   B operand: lane holds B[8g .. 8g+7][r]        (8 bf16)
//   D result : lane holds D[4g .. 4g+3][r]        (4 fp32)
// A 32-deep contraction may run over any fixed permutation of its index, as
// long as A and B use the same one.  The kernels use that freedom to feed a
// result straight back in as an operand: the D results of two consecutive
// 16-row blocks give, per lane, rows {4g..4g+3} and {16+4g..16+4g+3}, which is
// exactly what one operand needs if contraction index 8g+t stands for local
// row 4g+t (t < 4) or 16+4g+(t-4) (t >= 4).  chunk_row() is that map.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ inline f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// 16 bytes (8 bf16) from global or LDS memory, 16-byte aligned.
__device__ inline bf16x8 ld_bf16x8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// Two 8-byte pieces (4 bf16 each) joined into one operand.
__device__ inline bf16x8 ld_bf16x4x2(const uint16_t* lo, const uint16_t* hi) {
    u32x2 a = *reinterpret_cast<const u32x2*>(lo);
    u32x2 b = *reinterpret_cast<const u32x2*>(hi);
    u32x4 w = {a.x, a.y, b.x, b.y};
    return __builtin_bit_cast(bf16x8, w);
}

__device__ inline bf16x8 zero_bf16x8() { return __builtin_bit_cast(bf16x8, u32x4{0u, 0u, 0u, 0u}); }

// Round-to-nearest-even fp32 -> bf16 of two D results, as one operand.
__device__ inline bf16x8 pack_bf16x8(f32x4 lo, f32x4 hi) {
    bf16x4 a = __builtin_convertvector(lo, bf16x4);
    bf16x4 b = __builtin_convertvector(hi, bf16x4);
    return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__device__ inline uint2 pack_bf16x4_bits(f32x4 v) {
    bf16x4 a = __builtin_convertvector(v, bf16x4);
    return __builtin_bit_cast(uint2, a);
}

__device__ inline uint16_t bf16_bits(float x) {
    return __builtin_bit_cast(uint16_t, (__bf16)x);
}

__device__ inline float bf16_to_f32(uint16_t b) {
    return __uint_as_float((uint32_t)b << 16);
}

// Local row of contraction index 8g + t in a 32-row chunk (see top comment).
__device__ inline int chunk_row(int g, int t) { return t < 4 ? 4 * g + t : 16 + 4 * g + (t - 4); }

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Max / sum over the four lanes that share r = lane % 16.
__device__ inline float max_over_g(float x) {
    x = fmaxf(x, __shfl_xor(x, 16));
    return fmaxf(x, __shfl_xor(x, 32));
}
__device__ inline float sum_over_g(float x) {
    x += __shfl_xor(x, 16);
    return x + __shfl_xor(x, 32);
}

}  // namespace sa
