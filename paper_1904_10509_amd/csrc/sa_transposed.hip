// Strided pattern, merged heads (A1 u A2 of Sec. 4.3, eq. mergedmat of
// Sec. 5.1), with the A2 part computed by transposition (Sec. 5.5: a stride
// of l becomes a local window once the positions are reordered by their
// residue mod l).
//
// The merged set of row i is the band A1 = {max(0, i - l) .. i} and the A2
// positions outside it, {i - k l : k >= 2}.  The two pieces are disjoint, so
// the softmax over their union is the log-sum-exp combination of a softmax
// over each:
//   band:  the block-sparse kernels over the strided A1 layout;
//   rest:  in residue class r (positions r + m l, m = 0 .. M - 1, M = n / l)
//          query m attends keys m' <= m - 2: dense causal attention once the
//          queries are shifted by two class steps.  The shift is a copy of Q
//          (and, for the backward, of O and dO) two l-rows up with a zero
//          tail, [b, h, n, d] like K and V, so that all of them are seen in
//          class order through one set of strides: (n d, d, l d) over
//          (b h, class r, step m).
// Forward: band -> O1, LSE1; rest -> O2, LSE2 (class order); merge.
// Backward: the gradient of each piece given the merged O and LSE (the
// attention weights of the union are exp(S - LSE) on either piece), summed.
// Padded queries of the shifted copy (the tail) get LSE = +inf in the
// backward, hence zero weights and no contribution.
#include <math.h>

#include "sa_internal.h"
#include "sa_mfma.h"

namespace sa {

namespace {

constexpr int kThreads = 256;

// 8 consecutive elements as fp32, and back.
__device__ inline void load8(const uint16_t* p, float* x) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(u[e] << 16);
        x[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
}
__device__ inline void load8(const float* p, float* x) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[e] = a[e];
        x[4 + e] = b[e];
    }
}
__device__ inline uint32_t bf16_bits(float f) {
    const __bf16 b = (__bf16)f;  // round to nearest even
    return (uint32_t)__builtin_bit_cast(uint16_t, b);
}
__device__ inline void store8(uint16_t* p, const float* x) {
    u32x4 u;
#pragma unroll
    for (int e = 0; e < 4; ++e) u[e] = bf16_bits(x[2 * e]) | (bf16_bits(x[2 * e + 1]) << 16);
    *reinterpret_cast<u32x4*>(p) = u;
}
__device__ inline void store8(float* p, const float* x) {
    f32x4 a, b;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        a[e] = x[e];
        b[e] = x[4 + e];
    }
    *reinterpret_cast<f32x4*>(p) = a;
    *reinterpret_cast<f32x4*>(p + 4) = b;
}

// dst[bh][t] = src[bh][t + shift] (t + shift < n), else 0; [bh][n][d]
// contiguous, one thread per 8 elements.
template <typename T>
__global__ void __launch_bounds__(kThreads)
shift_rows_kernel(const T* __restrict__ src, T* __restrict__ dst, int64_t rows, int64_t n, int d, int64_t shift) {
    const int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int chunks = d / 8;
    if (x >= rows * chunks) return;
    const int64_t row = x / chunks, t = row % n;
    const int c = (int)(x - row * chunks);
    float v[8];
    if (t + shift < n) {
        load8(src + (row + shift) * d + 8 * c, v);
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = 0.f;
    }
    store8(dst + row * d + 8 * c, v);
}

// Class-order row statistics of the shifted queries: dst[bh][r][m] =
// src[bh][r + (m + 2) l] for m + 2 < M, else +inf (no weight in the backward).
__global__ void __launch_bounds__(kThreads)
shift_lse_kernel(const float* __restrict__ src, float* __restrict__ dst, int64_t rows, int64_t n, int32_t l) {
    const int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (x >= rows) return;
    const int64_t bh = x / n, y = x % n, M = n / l;
    const int64_t r = y / M, m = y % M;
    const int64_t t = r + (m + 2) * l;
    dst[x] = t < n ? src[bh * n + t] : INFINITY;
}

// o, lse of the union from the band (o1, lse1, original order) and the rest
// (o2 in the shifted copy's rows, lse2 in class order): position i >= 2l
// takes row i - 2l of o2 and class entry (r, m - 2); below 2l the rest is
// empty.  One thread per 8 elements of a row.
template <typename T>
__global__ void __launch_bounds__(kThreads)
merge_kernel(const T* __restrict__ o1, const float* __restrict__ lse1, const T* __restrict__ o2,
             const float* __restrict__ lse2, T* __restrict__ o, float* __restrict__ lse, int64_t rows, int64_t n,
             int d, int32_t l) {
    const int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int chunks = d / 8;
    if (x >= rows * chunks) return;
    const int64_t row = x / chunks, i = row % n, bh = row / n, M = n / l;
    const int c = (int)(x - row * chunks);
    const float a = lse1[row];
    float b = -INFINITY;
    const int64_t t = i - 2 * (int64_t)l;
    if (t >= 0) b = lse2[bh * n + (t % l) * M + t / l];
    const float mx = fmaxf(a, b);
    const float wa = expf(a - mx), wb = b == -INFINITY ? 0.f : expf(b - mx);
    const float z = wa + wb;
    float v1[8], v2[8], out[8];
    load8(o1 + row * d + 8 * c, v1);
    if (t >= 0) {
        load8(o2 + (bh * n + t) * d + 8 * c, v2);
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v2[e] = 0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = (wa * v1[e] + wb * v2[e]) / z;
    store8(o + row * d + 8 * c, out);
    if (c == 0) lse[row] = mx + logf(z);
}

// dst[bh][i] += src[bh][i - shift] for i >= shift (fp32 sum, one rounding).
template <typename T>
__global__ void __launch_bounds__(kThreads)
add_shifted_kernel(T* __restrict__ dst, const T* __restrict__ src, int64_t rows, int64_t n, int d, int64_t shift) {
    const int64_t x = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const int chunks = d / 8;
    if (x >= rows * chunks) return;
    const int64_t row = x / chunks, i = row % n;
    const int c = (int)(x - row * chunks);
    if (i < shift) return;
    float a[8], b[8];
    load8(dst + row * d + 8 * c, a);
    load8(src + (row - shift) * d + 8 * c, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) a[e] += b[e];
    store8(dst + row * d + 8 * c, a);
}

// Dense causal layout of mq block rows in closed form: row qb holds key
// blocks 0 .. qb (FULL below the diagonal, MASKED on it), column kb holds
// query blocks kb .. mq - 1.  One thread per block row.
__global__ void __launch_bounds__(kThreads)
causal_layout_kernel(int32_t mq, int32_t* __restrict__ row_ptr, int32_t* __restrict__ col_idx,
                     uint8_t* __restrict__ kind, int32_t* __restrict__ col_ptr, int32_t* __restrict__ row_idx,
                     uint8_t* __restrict__ kind_t) {
    const int32_t x = (int32_t)(blockIdx.x * kThreads + threadIdx.x);
    if (x > mq) return;
    const int64_t xx = x;
    row_ptr[x] = (int32_t)(xx * (xx + 1) / 2);
    col_ptr[x] = (int32_t)(xx * mq - xx * (xx - 1) / 2);
    if (x == mq) return;
    const int64_t e = xx * (xx + 1) / 2;
    for (int32_t kb = 0; kb <= x; ++kb) {
        col_idx[e + kb] = kb;
        kind[e + kb] = kb < x ? TILE_FULL : TILE_MASKED;
    }
    const int64_t f = xx * mq - xx * (xx - 1) / 2;
    for (int32_t qb = x; qb < mq; ++qb) {
        row_idx[f + qb - x] = qb;
        kind_t[f + qb - x] = qb > x ? TILE_FULL : TILE_MASKED;
    }
}

unsigned groups(int64_t threads) { return (unsigned)((threads + kThreads - 1) / kThreads); }

}  // namespace

hipError_t causal_layout_launch(int32_t mq, int32_t* row_ptr, int32_t* col_idx, uint8_t* kind, int32_t* col_ptr,
                                int32_t* row_idx, uint8_t* kind_t, hipStream_t stream) {
    hipLaunchKernelGGL(causal_layout_kernel, dim3(groups((int64_t)mq + 1)), dim3(kThreads), 0, stream, mq, row_ptr,
                       col_idx, kind, col_ptr, row_idx, kind_t);
    return hipGetLastError();
}

hipError_t shift_rows_launch(int dtype, const void* src, void* dst, int64_t rows, int64_t n, int d, int64_t shift,
                             hipStream_t stream) {
    const unsigned g = groups(rows * (d / 8));
    if (dtype == 1)
        hipLaunchKernelGGL(shift_rows_kernel<uint16_t>, dim3(g), dim3(kThreads), 0, stream, (const uint16_t*)src,
                           (uint16_t*)dst, rows, n, d, shift);
    else
        hipLaunchKernelGGL(shift_rows_kernel<float>, dim3(g), dim3(kThreads), 0, stream, (const float*)src,
                           (float*)dst, rows, n, d, shift);
    return hipGetLastError();
}

hipError_t shift_lse_launch(const float* src, float* dst, int64_t rows, int64_t n, int32_t l, hipStream_t stream) {
    hipLaunchKernelGGL(shift_lse_kernel, dim3(groups(rows)), dim3(kThreads), 0, stream, src, dst, rows, n, l);
    return hipGetLastError();
}

hipError_t merge_launch(int dtype, const void* o1, const float* lse1, const void* o2, const float* lse2, void* o,
                        float* lse, int64_t rows, int64_t n, int d, int32_t l, hipStream_t stream) {
    const unsigned g = groups(rows * (d / 8));
    if (dtype == 1)
        hipLaunchKernelGGL(merge_kernel<uint16_t>, dim3(g), dim3(kThreads), 0, stream, (const uint16_t*)o1, lse1,
                           (const uint16_t*)o2, lse2, (uint16_t*)o, lse, rows, n, d, l);
    else
        hipLaunchKernelGGL(merge_kernel<float>, dim3(g), dim3(kThreads), 0, stream, (const float*)o1, lse1,
                           (const float*)o2, lse2, (float*)o, lse, rows, n, d, l);
    return hipGetLastError();
}

hipError_t add_shifted_launch(int dtype, void* dst, const void* src, int64_t rows, int64_t n, int d, int64_t shift,
                              hipStream_t stream) {
    const unsigned g = groups(rows * (d / 8));
    if (dtype == 1)
        hipLaunchKernelGGL(add_shifted_kernel<uint16_t>, dim3(g), dim3(kThreads), 0, stream, (uint16_t*)dst,
                           (const uint16_t*)src, rows, n, d, shift);
    else
        hipLaunchKernelGGL(add_shifted_kernel<float>, dim3(g), dim3(kThreads), 0, stream, (float*)dst,
                           (const float*)src, rows, n, d, shift);
    return hipGetLastError();
}

}  // namespace sa
