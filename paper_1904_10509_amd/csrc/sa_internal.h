// Internal declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>

#include "sa_mask.h"
#include "sa_pattern.h"

namespace sa {

constexpr float kLog2eHost = 1.4426950408889634f;

// Present blocks of one layout, counted on the host with the O(1) test.
int64_t layout_count_host(const Pattern& p, int64_t n, int64_t B);

hipError_t layout_launch(int64_t n, int32_t block, int32_t pattern, int32_t mode, int32_t sub, int64_t l,
                         int64_t c, int n_layouts, int32_t* row_ptr, int32_t* col_idx,
                         uint8_t* kind, int32_t* col_ptr, int32_t* row_idx, uint8_t* kind_t,
                         hipStream_t stream);

// Calls f(pattern, mode) with both as compile-time constants
// (std::integral_constant), so that kernels are specialised per pattern and
// head mode.
template <typename F>
inline hipError_t with_pattern_mode(int pattern, int mode, F&& f) {
    using S = std::integral_constant<int, STRIDED>;
    using X = std::integral_constant<int, FIXED>;
    using M0 = std::integral_constant<int, MODE_A1>;
    using M1 = std::integral_constant<int, MODE_A2>;
    using M2 = std::integral_constant<int, MODE_MERGED>;
    using M3 = std::integral_constant<int, MODE_INTERLEAVED>;
    if (pattern == STRIDED) {
        switch (mode) {
        case MODE_A1: return f(S{}, M0{});
        case MODE_A2: return f(S{}, M1{});
        case MODE_MERGED: return f(S{}, M2{});
        default: return f(S{}, M3{});
        }
    }
    switch (mode) {
    case MODE_A1: return f(X{}, M0{});
    case MODE_A2: return f(X{}, M1{});
    case MODE_MERGED: return f(X{}, M2{});
    default: return f(X{}, M3{});
    }
}

// Orders in which the dK / dV kernel takes its work.
enum { CLAIM_QUEUES = 0, CLAIM_ROUND_ROBIN = 1, CLAIM_SERPENTINE = 2, CLAIM_XCD_SERPENTINE = 3 };

// Which blocks a kernel walks:
//   WALK_LAYOUT  the present blocks of the layout;
//   WALK_BAND    of a strided layout with l a multiple of B, only the blocks of
//                the band A1 = {i - l .. i}: the last l / B + 1 entries of a
//                row, the first l / B + 1 of a column (they hold no other
//                pair of the merged set);
//   WALK_DENSE   every block kb <= qb, without a layout (dense causal).
enum { WALK_LAYOUT = 0, WALK_BAND = 1, WALK_DENSE = 2 };

// What a kernel does with its result:
//   EPI_STORE  writes it;
//   EPI_MERGE  (forward) combines it, by log-sum-exp, with the O and LSE
//              already in the outputs (a softmax over a disjoint part of
//              each row's set);
//   EPI_ADD    (dQ, dK, dV) adds it to the gradient already in the output.
enum { EPI_STORE = 0, EPI_MERGE = 1, EPI_ADD = 2 };

// Everything a kernel needs to know about one call.
struct AttnArgs {
    int32_t pattern, mode;
    int32_t l, c;          // validated to fit in 32 bits
    int32_t n, nq, block;  // n < 2^31
    int32_t batch, heads, d;
    int64_t sb, sh, ss;    // element strides: batch, head, sequence
    float scale;           // softmax scale (> 0)
    float scale_log2;      // scale * log2(e)
    uint64_t period_bits;  // bits at multiples of l below 64 (strided masks)
    uint64_t sum_lo, sum_hi;  // summary positions below 128 (fixed masks, l <= 64, subblock 0)
    int32_t sub;           // fixed: 0 = one summary window for all heads, else floor(l / c) subblocks
    int32_t claim_mode;    // dK / dV work order, one of CLAIM_* (set by the backward launcher)
    int32_t pairs;         // dK / dV: summary halves walked in pairs (set by the backward launcher)
    int32_t row_stats;     // dQ: compute the row statistics itself, in place of the pre kernel (set by the launcher)
    DivL dl;               // division by l
    int32_t walk;          // WALK_*
    int32_t qshift;        // masks see query i as i - qshift (a causal limit j <= i - qshift)
    int32_t epilogue;      // EPI_*
    int64_t lse_sb, lse_sh, lse_ss;  // element strides of LSE and the row statistics (batch, head, row)
    const int32_t* row_ptr;
    const int32_t* col_idx;
    const uint8_t* kind;
    const int32_t* col_ptr;
    const int32_t* row_idx;
    const uint8_t* kind_t;
};

// The (head, query block, batch) of a row-view workgroup, on the grid
// (heads, nq, batch).  The dispatcher hands consecutive workgroups to the 8
// XCDs in turn, so workgroup L (x fastest) runs on XCD L mod 8.  A walk of
// every block (the residue classes, each a short dense problem read at a
// stride of l rows) gives the nq workgroups of one (batch, head) consecutive
// places s = L / 8 on one XCD: its keys then stay in that XCD's L2 while all
// its query blocks walk them, instead of leaving it between the query-block
// generations of the plain order.  Needs batch x heads a multiple of 8;
// otherwise, and for other walks, the plain order.  Longest rows first.
struct GridItem {
    int h, qb, b;
};
__device__ inline GridItem row_grid_item(const AttnArgs& a) {
    if (a.walk == WALK_DENSE && ((int64_t)a.batch * a.heads) % 8 == 0) {
        const uint64_t L = blockIdx.x + (uint64_t)gridDim.x * (blockIdx.y + (uint64_t)gridDim.y * blockIdx.z);
        const uint64_t s = L / 8;
        const uint64_t u = (s / (uint64_t)a.nq) * 8 + L % 8;  // (batch, head) unit
        return {(int)(u % (uint64_t)a.heads), a.nq - 1 - (int)(s % (uint64_t)a.nq), (int)(u / (uint64_t)a.heads)};
    }
    return {(int)blockIdx.x, a.nq - 1 - (int)blockIdx.y, (int)blockIdx.z};
}

// Index of row i of (batch b, head h) in LSE and the backward's row statistics.
__host__ __device__ inline int64_t stat_index(const AttnArgs& a, int b, int h, int64_t i) {
    return (int64_t)b * a.lse_sb + (int64_t)h * a.lse_sh + i * a.lse_ss;
}

// Layout that head h reads.
__host__ __device__ inline int head_layout(const AttnArgs& a, int h) { return layout_of_head(a.mode, a.sub, h); }

// First summary position of subblock s inside an l-block (fixed pattern).
__host__ __device__ inline int32_t window_start(const AttnArgs& a, int s) {
    return (int32_t)summary_start(a.l, a.c, s);
}

// Mask parameters of one part and summary subblock s.  With distinct
// subblocks and l <= 64 the 128-position summary words are built here (a few
// scalar steps per workgroup); otherwise they come with the call.
__device__ inline MaskParams mask_params(const AttnArgs& a, int pattern, int part, int s) {
    MaskParams mp{pattern, part, a.l, a.c, a.period_bits, a.sum_lo, a.sum_hi, window_start(a, s)};
    if (pattern == FIXED && s != 0 && a.l <= 64) summary_words(a.l, a.c, mp.w, &mp.sum_lo, &mp.sum_hi);
    return mp;
}
__device__ inline MaskParams head_mask_params(const AttnArgs& a, int pattern, int mode, int h) {
    return mask_params(a, pattern, part_of_head(mode, h), subblock_of_head(a.sub, h));
}

// Forward.  q, k, v, o use the strides in `a`; lse is [batch, heads, n].
hipError_t fwd_launch(const AttnArgs& a, int dtype, const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream);

// Backward workspace: D and the base-2 LSE per row [b, h, n] (fp32), then
// the work queues and the column order of the dK / dV kernel.
// Whether the row-view kernels (forward, dQ) carry a second step body for
// fully attended blocks: always in the fixed pattern and for walks of the band
// or of every block (l / B - 1 of a band row's l / B + 1 blocks are full, and
// all but the diagonal of a dense row); over a strided layout when those
// blocks (l / B - 1 per row) outnumber the diagonal-only blocks of a middle
// row (about n / 2l), i.e. 2 l^2 > n B, as in the dense limit l >= n.
// Otherwise the second copy of the code costs more than it saves.
template <int PAT, typename F>
inline hipError_t with_full_body(const AttnArgs& a, F&& f) {
    if constexpr (PAT == FIXED) {
        return f(std::true_type{});
    } else {
        if (a.walk != WALK_LAYOUT || 2.0 * (double)a.l * (double)a.l > (double)a.n * (double)a.block)
            return f(std::true_type{});
        return f(std::false_type{});
    }
}

size_t decode_workspace_bytes(int pattern, int mode, int32_t sub, int32_t pos, int32_t l, int32_t c,
                              int64_t batch, int64_t heads, int d);
hipError_t decode_launch(int pattern, int mode, int32_t sub, int32_t pos, int32_t l, int32_t c, int batch, int heads,
                         int d, int dtype, const void* q, const int64_t* q_strides, const void* k, const void* v,
                         const int64_t* kv_strides, float scale, void* o, float* lse, void* workspace,
                         hipStream_t stream);

size_t bwd_workspace_bytes(int64_t batch, int64_t heads, int64_t n, int64_t nq, int n_layouts);

// Launches of a backward call: the row statistics (pre), dQ, and dK / dV.
enum { BWD_PRE = 1, BWD_DQ = 2, BWD_DKDV = 4, BWD_ALL = 7 };

// Backward; `parts` selects its launches.
hipError_t bwd_launch(const AttnArgs& a, int dtype, const void* q, const void* k, const void* v,
                      const void* o, const void* dout, const float* lse, void* dq, void* dk,
                      void* dv, void* workspace, hipStream_t stream, int parts = BWD_ALL);

}  // namespace sa
