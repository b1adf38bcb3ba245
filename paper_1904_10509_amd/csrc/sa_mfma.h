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
// row 4g+t (t < 4) or 16+4g+(t-4) (t >= 4): pack_bf16x8 of the two results.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

__device__ inline f32x4 mfma_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// 16 bytes (8 bf16) from global or LDS memory, 16-byte aligned.
__device__ inline bf16x8 ld_bf16x8(const uint16_t* p) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// The same from global memory with a non-temporal load, for data read once
// that should not displace lines other workgroups still share.
__device__ inline bf16x8 ld_bf16x8_once(const uint16_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const bf16x8*>(p));
}

// Round-to-nearest-even fp32 -> bf16 of two D results, as one operand.
__device__ inline bf16x8 pack_bf16x8(f32x4 lo, f32x4 hi) {
    bf16x4 a = __builtin_convertvector(lo, bf16x4);
    bf16x4 b = __builtin_convertvector(hi, bf16x4);
    return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// The same two results as a high and a low operand: hi = bf16(x) and
// lo = bf16(x - hi), so that hi + lo carries x to about 2^-16 of itself
// where hi alone carries it to 2^-8.
__device__ inline void split_bf16x8(f32x4 a, f32x4 b, bf16x8& hi, bf16x8& lo) {
    hi = pack_bf16x8(a, b);
    f32x4 ra, rb;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        ra[t] = a[t] - (float)hi[t];
        rb[t] = b[t] - (float)hi[4 + t];
    }
    lo = pack_bf16x8(ra, rb);
}

__device__ inline uint2 pack_bf16x4_bits(f32x4 v) {
    bf16x4 a = __builtin_convertvector(v, bf16x4);
    return __builtin_bit_cast(uint2, a);
}

// Four bf16 (8 bytes) to fp32, exactly.
__device__ inline f32x4 bf16x4_to_f32x4(uint2 u) {
    return f32x4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                 __uint_as_float(u.y & 0xffff0000u)};
}

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// sum_e a[e] b[e] over 8 bf16 pairs in fp32: four v_dot2_f32_bf16 on two
// independent accumulators (a dependency chain of two, not eight).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ inline float dot_bf16x8(bf16x8 a, bf16x8 b) {
    const bf16x2 a0{a[0], a[1]}, a1{a[2], a[3]}, a2{a[4], a[5]}, a3{a[6], a[7]};
    const bf16x2 b0{b[0], b[1]}, b1{b[2], b[3]}, b2{b[4], b[5]}, b3{b[6], b[7]};
    float x = __builtin_amdgcn_fdot2_f32_bf16(a0, b0, 0.f, false);
    float y = __builtin_amdgcn_fdot2_f32_bf16(a1, b1, 0.f, false);
    x = __builtin_amdgcn_fdot2_f32_bf16(a2, b2, x, false);
    y = __builtin_amdgcn_fdot2_f32_bf16(a3, b3, y, false);
    return x + y;
}

// Max / sum over the four lanes that share r = lane % 16, with the gfx950
// row-swap permutes (16-lane rows 0<->1, 2<->3, then the two 32-lane halves).
__device__ inline float max_over_g(float x) {
    auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ inline float sum_over_g(float x) {
    auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Transposing LDS read (ds_read_b64_tr_b16).  Within each 16-lane row of the
// wave, output lane i receives element (i mod 4) of the 8 bytes addressed by
// input lane 4u + i/4, as its item u (u = 0..3).  Issue it with every lane
// active: under a partial exec mask the inactive lanes' destination registers
// did not keep their old contents in testing.  So if lane L of the row
// points at &T[row0 + L/4][col0 + 4 (L mod 4)] of a row-major bf16 tile T,
// lane i receives T[row0 + u][col0 + i] for u = 0..3: four rows of one column.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ inline u32x2 ld_tr16(const uint16_t* lds_ptr) {
    s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(lds_ptr));
    return __builtin_bit_cast(u32x2, v);
}

}  // namespace sa
