// Pattern math of the library (host and device): block presence in O(1),
// attended-pair counts over a column range in O(1), and the element predicate
// used to mask partial blocks.  Sets are those of Sec. 4.3 (0-based, causal);
// the closed forms below are derived from them.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

enum { STRIDED = 0, FIXED = 1 };
enum { MODE_A1 = 0, MODE_A2 = 1, MODE_MERGED = 2, MODE_INTERLEAVED = 3 };
enum { PART_A1 = 0, PART_A2 = 1, PART_MERGED = 2 };
enum { TILE_FULL = 0, TILE_MASKED = 1 };

struct Pattern {
    int32_t pattern;  // STRIDED or FIXED
    int32_t part;     // PART_A1, PART_A2 or PART_MERGED
    int64_t l;        // stride
    int64_t c;        // summary width (fixed pattern)
    int64_t w;        // first summary position inside an l-block (fixed pattern)
};

// Factor a head uses (Sec. 5.1).
__host__ __device__ inline int part_of_head(int mode, int h) {
    if (mode == MODE_INTERLEAVED) return (h & 1) ? PART_A2 : PART_A1;
    return mode == MODE_A1 ? PART_A1 : (mode == MODE_A2 ? PART_A2 : PART_MERGED);
}

// Part held by layout g.
__host__ __device__ inline int part_of_layout(int mode, int g) {
    if (mode == MODE_INTERLEAVED) return g == 0 ? PART_A1 : PART_A2;
    return part_of_head(mode, 0);
}

// Summary subblocks (Sec. 4.3, closing remark on the fixed pattern: heads may
// attend different c-wide subblocks of each l-block).  `sub` = 0: every head
// uses the last c positions of each block.  sub = floor(l / c) > 0: subblock
// s, numbered from the end of the block, holds positions l - (s + 1) c ..
// l - s c - 1, and head h uses s = h mod sub.  Layouts, one per distinct set:
// A1 alone 1; A2 or merged `sub`, layout s for subblock s; alternating heads
// 1 + sub, layout 0 for A1 and 1 + s for A2 with subblock s.
__host__ __device__ inline int64_t summary_start(int64_t l, int64_t c, int64_t s) { return l - (s + 1) * c; }

__host__ __device__ inline int layout_count(int mode, int sub) {
    if (sub == 0 || mode == MODE_A1) return mode == MODE_INTERLEAVED ? 2 : 1;
    return mode == MODE_INTERLEAVED ? 1 + sub : sub;
}
__host__ __device__ inline int subblock_of_head(int sub, int h) { return sub > 0 ? h % sub : 0; }
__host__ __device__ inline int layout_of_head(int mode, int sub, int h) {
    if (mode == MODE_INTERLEAVED) return (h & 1) ? 1 + subblock_of_head(sub, h) : 0;
    return mode == MODE_A1 ? 0 : subblock_of_head(sub, h);
}
__host__ __device__ inline int subblock_of_layout(int mode, int sub, int g) {
    if (sub == 0 || mode == MODE_A1) return 0;
    return mode == MODE_INTERLEAVED ? (g == 0 ? 0 : g - 1) : g;
}

__host__ __device__ inline int64_t min64(int64_t a, int64_t b) { return a < b ? a : b; }
__host__ __device__ inline int64_t max64(int64_t a, int64_t b) { return a > b ? a : b; }

// First fixed-pattern summary column >= x (x >= 0); the summary columns are
// the positions w .. w + c - 1 of every l-block.
__host__ __device__ inline int64_t first_summary_at_or_after(int64_t x, int64_t l, int64_t c, int64_t w) {
    const int64_t r = x % l;
    if (r < w) return x - r + w;
    return r < w + c ? x : x - r + l + w;
}

// Is any pair of the block rows [r0, r1] x columns [c0, c1] attended?  The
// caller guarantees c0 <= r1 (blocks on or below the diagonal).
__host__ __device__ inline bool block_present_part(int pattern, int part, int64_t l, int64_t c, int64_t w,
                                                   int64_t r0, int64_t r1, int64_t c0, int64_t c1) {
    if (pattern == STRIDED) {
        int64_t dmin = r0 - c1, dmax = r1 - c0;  // every difference i - j in between occurs
        if (part == PART_A1) return dmin <= l;
        // a multiple of l in [max(0, dmin), dmax]
        return (dmax / l) * l >= max64(0, dmin);
    }
    if (part == PART_A1) {
        // some l-block meets both the rows and the columns
        return max64(r0 / l, c0 / l) <= min64(r1 / l, c1 / l);
    }
    return first_summary_at_or_after(c0, l, c, w) <= min64(c1, r1);
}

__host__ __device__ inline bool block_present(const Pattern& p, int64_t r0, int64_t r1, int64_t c0,
                                              int64_t c1) {
    if (p.part == PART_MERGED)
        return block_present_part(p.pattern, PART_A1, p.l, p.c, p.w, r0, r1, c0, c1) ||
               block_present_part(p.pattern, PART_A2, p.l, p.c, p.w, r0, r1, c0, c1);
    return block_present_part(p.pattern, p.part, p.l, p.c, p.w, r0, r1, c0, c1);
}

// Number of integers in [lo, hi].
__host__ __device__ inline int64_t span(int64_t lo, int64_t hi) { return hi >= lo ? hi - lo + 1 : 0; }

// Number of j in [lo, hi] with j = i - k*l, k >= 0 (0 <= lo, hi <= i).
__host__ __device__ inline int64_t strided_hits(int64_t i, int64_t l, int64_t lo, int64_t hi) {
    if (hi < lo) return 0;
    int64_t kmax = (i - lo) / l;
    int64_t kmin = (i - hi + l - 1) / l;
    return kmax >= kmin ? kmax - kmin + 1 : 0;
}

// Number of summary columns in [0, x] (x >= -1).
__host__ __device__ inline int64_t summary_upto(int64_t x, int64_t l, int64_t c, int64_t w) {
    int64_t m = x + 1;
    return (m / l) * c + min64(c, max64(0, m % l - w));
}

// |S_i intersected with [lo, hi]| for one part (lo >= 0).
__host__ __device__ inline int64_t attended_in_range(const Pattern& p, int64_t i, int64_t lo,
                                                     int64_t hi) {
    hi = min64(hi, i);
    if (hi < lo) return 0;
    if (p.pattern == STRIDED) {
        int64_t band = span(max64(lo, i - p.l), hi);
        if (p.part == PART_A1) return band;
        if (p.part == PART_A2) return strided_hits(i, p.l, lo, hi);
        return band + strided_hits(i, p.l, lo, min64(hi, i - p.l - 1));
    }
    int64_t blk0 = (i / p.l) * p.l;
    int64_t own = span(max64(lo, blk0), hi);
    if (p.part == PART_A1) return own;
    if (p.part == PART_A2) return summary_upto(hi, p.l, p.c, p.w) - summary_upto(lo - 1, p.l, p.c, p.w);
    int64_t hi2 = min64(hi, blk0 - 1);
    int64_t earlier = hi2 >= lo ? summary_upto(hi2, p.l, p.c, p.w) - summary_upto(lo - 1, p.l, p.c, p.w) : 0;
    return own + earlier;
}

// True when every pair of the block rows [r0, r1] x columns [c0, c1] is
// attended, evaluated in O(1) on the scalar unit by the kernels (the layout
// builder counts pairs instead).  Exact for every part except fixed merged,
// where it may answer false for a full block, which only costs masking work.
__host__ __device__ inline bool block_full(int pattern, int part, int64_t l, int64_t c, int64_t w, int64_t r0,
                                           int64_t r1, int64_t c0, int64_t c1) {
    if (r0 < c1) return false;  // meets the diagonal: the causal cut runs through it
    if (pattern == STRIDED) {
        if (part == PART_A2) return l == 1;
        return r1 - c0 <= l || (part == PART_MERGED && l == 1);
    }
    const bool one_block = c0 / l == r1 / l;                                   // all pairs in one l-block
    const bool all_summary =  // every column a summary
        c == l || (c0 / l == c1 / l && c0 % l >= w && c1 % l < w + c);
    if (part == PART_A1) return one_block;
    if (part == PART_A2) return all_summary;
    return one_block || all_summary;
}

// Division by the stride l for 0 <= x < 2^31 with one 32 x 32 -> 64-bit
// multiply: with s = ceil(log2 l) and m = ceil(2^(31+s) / l) <= 2^31 (< 2^32),
// floor(x / l) equals floor(x m / 2^(31+s)), because m l - 2^(31+s) < l makes
// the error term x (m l - 2^(31+s)) / (l 2^(31+s)) smaller than 2^-s <= 1/l.
// (l = 1 gives m = 2^31 and the identity.)
struct DivL {
    int32_t l;
    int32_t shift;  // 31 + ceil(log2 l)
    uint32_t m;
};

inline DivL make_divl(int32_t l) {
    int s = 0;
    while ((1ll << s) < l) ++s;
    DivL d{l, 31 + s, (uint32_t)(((1ull << (31 + s)) + (uint64_t)l - 1) / (uint64_t)l)};
    return d;
}

__host__ __device__ inline int32_t div_l(const DivL& d, int32_t x) {
    return (int32_t)(((uint64_t)(uint32_t)x * d.m) >> d.shift);
}
__host__ __device__ inline int32_t mod_l(const DivL& d, int32_t x) { return x - div_l(d, x) * d.l; }

// block_full in 32-bit arithmetic (all coordinates below 2^31).
__host__ __device__ inline bool block_full32(int pattern, int part, const DivL& dl, int32_t c, int32_t w, int32_t r0,
                                             int32_t r1, int32_t c0, int32_t c1) {
    const int32_t l = dl.l;
    if (r0 < c1) return false;
    if (pattern == STRIDED) {
        if (part == PART_A2) return l == 1;
        return r1 - c0 <= l || (part == PART_MERGED && l == 1);
    }
    const int32_t c0_blk = div_l(dl, c0);
    const bool one_block = c0_blk == div_l(dl, r1);
    const bool all_summary =
        c == l || (c0_blk == div_l(dl, c1) && c0 - c0_blk * l >= w && c1 - c0_blk * l < w + c);
    if (part == PART_A1) return one_block;
    if (part == PART_A2) return all_summary;
    return one_block || all_summary;
}

// The set S_pos of one query position (Sec. 4.3) as an index space for
// decoding: key t (0 <= t < count) is position at(t), each position of the set
// exactly once.  Order: the A1 interval ascending, then the A2 positions
// outside it (strided: pos - 2l, pos - 3l, ...; fixed: the summary columns of
// the earlier l-blocks, ascending).  A2 alone: strided pos, pos - l, ...;
// fixed the summary columns up to pos, ascending.  dc divides by c; the
// summary columns are the positions w .. w + c - 1 of every l-block (fixed).
struct DecodeSet {
    int pattern, part;
    int32_t pos, l, c, w;
    int32_t a1_lo;      // A1 is [a1_lo, a1_lo + n1)
    int64_t n1;         // up to 2^31 (pos = 2^31 - 1 with A1 from 0)
    int64_t count;
    DivL dc;
    __host__ __device__ DecodeSet(int pattern_, int part_, int32_t pos_, int32_t l_, int32_t c_, int32_t w_,
                                  const DivL& dc_)
        : pattern(pattern_), part(part_), pos(pos_), l(l_), c(c_), w(w_), dc(dc_) {
        const int32_t lblk = pos / l;
        if (pattern == STRIDED) {
            a1_lo = pos - l > 0 ? pos - l : 0;
            n1 = (int64_t)pos - a1_lo + 1;
            if (part == PART_A1) count = n1;
            else if (part == PART_A2) count = (int64_t)lblk + 1;
            else count = n1 + (lblk > 1 ? lblk - 1 : 0);
        } else {
            a1_lo = lblk * l;
            n1 = (int64_t)pos - a1_lo + 1;
            const int32_t first_sum = a1_lo + w;  // first summary column of pos's l-block
            const int32_t own = pos >= first_sum ? (pos - first_sum + 1 < c ? pos - first_sum + 1 : c) : 0;
            if (part == PART_A1) count = n1;
            else if (part == PART_A2) count = (int64_t)lblk * c + own;
            else count = n1 + (int64_t)lblk * c;
        }
    }
    __host__ __device__ int32_t summary(int32_t u) const {  // u-th summary column from position 0
        const int32_t blk = div_l(dc, u);
        return blk * l + w + (u - blk * c);
    }
    __host__ __device__ int32_t at(int64_t t) const {
        if (pattern == STRIDED) {
            if (part == PART_A2) return pos - (int32_t)t * l;
            if (t < n1) return a1_lo + (int32_t)t;
            return pos - ((int32_t)(t - n1) + 2) * l;
        }
        if (part == PART_A2) return summary((int32_t)t);
        if (t < n1) return a1_lo + (int32_t)t;
        return summary((int32_t)(t - n1));
    }
};

// Element predicate in 32-bit arithmetic (0 <= i, j < 2^31).
__host__ __device__ inline bool attended(int pattern, int part, int32_t l, int32_t c, int32_t w, int32_t i,
                                         int32_t j) {
    if (j > i) return false;
    if (pattern == STRIDED) {
        int32_t d = i - j;
        bool a1 = d <= l;
        bool a2 = (d % l) == 0;
        return part == PART_A1 ? a1 : (part == PART_A2 ? a2 : (a1 || a2));
    }
    bool a1 = (i / l) == (j / l);
    const int32_t r = j % l;
    bool a2 = r >= w && r < w + c;
    return part == PART_A1 ? a1 : (part == PART_A2 ? a2 : (a1 || a2));
}

}  // namespace sa
