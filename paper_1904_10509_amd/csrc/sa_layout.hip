// Block layout builder (Sec. 5.5: the product is computed over B x B blocks and
// blocks above the diagonal are never visited).
//
// Three launches on the caller's stream:
//   1. count:  one wave per (layout g, index x) counts the present blocks of
//              query-block row x and of key-block column x (O(1) test each);
//   2. scan:   one workgroup turns the counts into absolute CSR offsets for
//              both views at once;
//   3. fill:   one wave per (g, x) writes row x (ascending key blocks) and
//              column x (ascending query blocks) using ballots for positions,
//              and classifies each present block as FULL or MASKED by counting
//              its attended pairs in closed form (O(B) per block).
// Row and column views are produced independently (no atomics), so the
// result is deterministic.
#include "sa_internal.h"
#include "sa_pattern.h"

namespace sa {

namespace {

constexpr int kWave = 64;

__device__ inline uint64_t lanes_below(int lane) {
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

struct LayoutArgs {
    int64_t nq;
    int32_t block;
    int32_t pattern;
    int32_t mode;
    int32_t sub;  // summary subblocks (0: one window for all heads)
    int64_t l, c;
};

__device__ inline Pattern pattern_of(const LayoutArgs& a, int g) {
    Pattern p;
    p.pattern = a.pattern;
    p.part = part_of_layout(a.mode, g);
    p.l = a.l;
    p.c = a.c;
    p.w = summary_start(a.l, a.c, subblock_of_layout(a.mode, a.sub, g));
    return p;
}

__device__ inline bool present(const Pattern& p, int64_t B, int64_t qb, int64_t kb) {
    return block_present(p, qb * B, qb * B + B - 1, kb * B, kb * B + B - 1);
}

__device__ inline uint8_t block_kind(const Pattern& p, int64_t B, int64_t qb, int64_t kb) {
    int64_t c0 = kb * B, c1 = c0 + B - 1, total = 0;
    for (int64_t i = qb * B; i < qb * B + B; ++i) total += attended_in_range(p, i, c0, c1);
    return total == B * B ? TILE_FULL : TILE_MASKED;
}

// grid: (nq, n_layouts), block: 64 threads (one wave).
__global__ void __launch_bounds__(kWave) layout_count_kernel(LayoutArgs a, int32_t* row_ptr,
                                                             int32_t* col_ptr) {
    const int g = blockIdx.y;
    const int64_t x = blockIdx.x;
    const int lane = threadIdx.x;
    const int64_t B = a.block;
    Pattern p = pattern_of(a, g);
    int64_t rows = 0, cols = 0;
    for (int64_t kb = lane; kb <= x; kb += kWave) rows += present(p, B, x, kb);
    for (int64_t qb = x + lane; qb < a.nq; qb += kWave) cols += present(p, B, qb, x);
    for (int off = 32; off > 0; off >>= 1) {
        rows += __shfl_xor(rows, off);
        cols += __shfl_xor(cols, off);
    }
    if (lane == 0) {
        int64_t base = (int64_t)g * (a.nq + 1);
        row_ptr[base + x + 1] = (int32_t)rows;
        col_ptr[base + x + 1] = (int32_t)cols;
        if (x == 0) {
            row_ptr[base] = 0;
            col_ptr[base] = 0;
        }
    }
}

// In-place inclusive scan of `len` int32 counts (the leading zero of each
// layout makes the result absolute CSR offsets).  One workgroup of 1024.
constexpr int kScanThreads = 1024;

__device__ void block_inclusive_scan(int32_t* data, int64_t len) {
    __shared__ int64_t partial[kScanThreads];
    const int t = threadIdx.x;
    const int64_t per = (len + kScanThreads - 1) / kScanThreads;
    const int64_t lo = min64(len, (int64_t)t * per), hi = min64(len, lo + per);
    int64_t sum = 0;
    for (int64_t e = lo; e < hi; ++e) sum += data[e];
    partial[t] = sum;
    __syncthreads();
    for (int off = 1; off < kScanThreads; off <<= 1) {
        int64_t v = t >= off ? partial[t - off] : 0;
        __syncthreads();
        partial[t] += v;
        __syncthreads();
    }
    int64_t run = t > 0 ? partial[t - 1] : 0;
    for (int64_t e = lo; e < hi; ++e) {
        run += data[e];
        data[e] = (int32_t)run;
    }
    __syncthreads();
}

__global__ void __launch_bounds__(kScanThreads) layout_scan_kernel(int32_t* row_ptr,
                                                                   int32_t* col_ptr, int64_t len) {
    block_inclusive_scan(row_ptr, len);
    block_inclusive_scan(col_ptr, len);
}

// grid: (nq, n_layouts), block: one wave.
__global__ void __launch_bounds__(kWave) layout_fill_kernel(LayoutArgs a, const int32_t* row_ptr,
                                                            int32_t* col_idx, uint8_t* kind,
                                                            const int32_t* col_ptr,
                                                            int32_t* row_idx, uint8_t* kind_t) {
    const int g = blockIdx.y;
    const int64_t x = blockIdx.x;
    const int lane = threadIdx.x;
    const int64_t B = a.block;
    Pattern p = pattern_of(a, g);
    const int64_t base = (int64_t)g * (a.nq + 1);

    int64_t pos = row_ptr[base + x];
    for (int64_t k0 = 0; k0 <= x; k0 += kWave) {
        int64_t kb = k0 + lane;
        bool on = kb <= x && present(p, B, x, kb);
        uint64_t mask = __ballot(on);
        if (on) {
            int64_t e = pos + __popcll(mask & lanes_below(lane));
            col_idx[e] = (int32_t)kb;
            kind[e] = block_kind(p, B, x, kb);
        }
        pos += __popcll(mask);
    }

    pos = col_ptr[base + x];
    for (int64_t q0 = x; q0 < a.nq; q0 += kWave) {
        int64_t qb = q0 + lane;
        bool on = qb < a.nq && present(p, B, qb, x);
        uint64_t mask = __ballot(on);
        if (on) {
            int64_t e = pos + __popcll(mask & lanes_below(lane));
            row_idx[e] = (int32_t)qb;
            kind_t[e] = block_kind(p, B, qb, x);
        }
        pos += __popcll(mask);
    }
}

}  // namespace

int64_t layout_count_host(const Pattern& p, int64_t n, int64_t B) {
    const int64_t nq = n / B;
    int64_t total = 0;
    for (int64_t qb = 0; qb < nq; ++qb)
        for (int64_t kb = 0; kb <= qb; ++kb)
            total += block_present(p, qb * B, qb * B + B - 1, kb * B, kb * B + B - 1);
    return total;
}

hipError_t layout_launch(int64_t n, int32_t block, int32_t pattern, int32_t mode, int32_t sub, int64_t l,
                         int64_t c, int n_layouts, int32_t* row_ptr, int32_t* col_idx,
                         uint8_t* kind, int32_t* col_ptr, int32_t* row_idx, uint8_t* kind_t,
                         hipStream_t stream) {
    LayoutArgs a;
    a.nq = n / block;
    a.block = block;
    a.pattern = pattern;
    a.mode = mode;
    a.sub = sub;
    a.l = l;
    a.c = c;
    dim3 grid((unsigned)a.nq, (unsigned)n_layouts);
    hipLaunchKernelGGL(layout_count_kernel, grid, dim3(kWave), 0, stream, a, row_ptr, col_ptr);
    hipLaunchKernelGGL(layout_scan_kernel, dim3(1), dim3(kScanThreads), 0, stream, row_ptr,
                       col_ptr, (int64_t)n_layouts * (a.nq + 1));
    hipLaunchKernelGGL(layout_fill_kernel, grid, dim3(kWave), 0, stream, a, row_ptr, col_idx,
                       kind, col_ptr, row_idx, kind_t);
    return hipGetLastError();
}

}  // namespace sa
