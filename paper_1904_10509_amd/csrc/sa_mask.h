// Attended-position bitmasks for partial (MASKED) blocks.
//
// Inside a B x B block each lane owns either one query row (forward) or one
// key column (backward).  Instead of evaluating the element predicate of the
// sets of Sec. 4.3 per element, the lane builds once per block a 64-bit mask
// of the attended positions along its row or column, from a few interval and
// periodic patterns:
//   causal            j <= i
//   strided A1        i - l <= j              (an interval)
//   strided A2        i - j == 0 mod l        (bits at a period of l)
//   fixed A1          same l-block            (an interval)
//   fixed A2          w <= j mod l < w + c    (c-wide runs at a period of l;
//                                             w = l - c unless heads have
//                                             their own subblocks)
// Elements then test one bit each.
#pragma once

#include <stdint.h>

#include "sa_pattern.h"

namespace sa {

// Bits lo..hi of a 64-bit word (empty when hi < lo); lo, hi may lie outside
// [0, 63].  Written with selects only, so per-lane bounds cause no branch.
__device__ inline uint64_t bit_range(int lo, int hi) {
    const uint64_t upper = hi < 0 ? 0ull : (~0ull >> (63 - (hi > 63 ? 63 : hi)));
    const uint64_t lower = lo > 63 ? 0ull : (~0ull << (lo < 0 ? 0 : lo));
    return upper & lower;
}

// Bits at positions m, m + l, m + 2l, ... below 64, from `period_bits`
// (bits at 0, l, 2l, ... precomputed for the call).
__device__ inline uint64_t periodic_from(uint64_t period_bits, int m) {
    return (unsigned)m >= 64u ? 0ull : (period_bits << m);  // m < 0 (never used) also gives 0
}

// Non-negative remainder.
__device__ inline int mod_pos(int x, int l) {
    int r = x % l;
    return r < 0 ? r + l : r;
}

struct MaskParams {
    int pattern, part, l, c;
    uint64_t period_bits;  // strided: bits at multiples of l below 64
    uint64_t sum_lo, sum_hi;  // fixed, l <= 64: summary positions p < 128 (w <= p mod l < w + c)
    int w;                 // fixed: first summary position inside an l-block
};

// Summary columns (w <= j mod l < w + c) among j0 .. j0 + 63, as bits over
// j - j0; r0 = j0 mod l.  For l <= 64 it is the precomputed 128-position
// pattern shifted by r0; for l > 64 the runs start at w - r0 + k l, and only
// k = 0 (which may begin before j0) and k = 1 reach the 64 positions (k = -1
// ends at w + c - 1 - r0 - l < 0, k = 2 starts past 2l - r0 > l > 64).
// Wave-uniform arguments: evaluated on the scalar unit.
__device__ inline uint64_t summary_bits(const MaskParams& p, int r0) {
    if (p.l <= 64) return r0 == 0 ? p.sum_lo : (p.sum_lo >> r0) | (p.sum_hi << (64 - r0));
    const int s = p.w - r0;
    return bit_range(s, s + p.c - 1) | bit_range(s + p.l, s + p.l + p.c - 1);
}

// Bits of the 32-row (or 32-column) chunk qc of a lane's mask after the
// lane's shift by 4 (lane / 16): items 16 q + t, q = 2 qc, 2 qc + 1, t < 4.
__device__ inline uint32_t chunk_bits(uint64_t bits, int qc, bool two_blocks) {
    return (uint32_t)(bits >> (32 * qc)) & (two_blocks ? 0x000F000Fu : 0x0000000Fu);
}

// How a chunk (32 queries or keys of one 16-wide block of the other side)
// is treated, decided for the whole wave: nothing attended (no exponentials,
// zero probabilities), everything attended (no masking), or per item.
enum { CHUNK_NONE = 0, CHUNK_PART = 1, CHUNK_ALL = 2 };

__device__ inline int chunk_class(uint32_t lane_bits, bool two_blocks) {
    const uint32_t full = two_blocks ? 0x000F000Fu : 0x0000000Fu;
    const uint64_t any = __builtin_amdgcn_ballot_w64(lane_bits != 0u);
    const uint64_t short_of_full = __builtin_amdgcn_ballot_w64(lane_bits != full);
    return any == 0ull ? CHUNK_NONE : (short_of_full == 0ull ? CHUNK_ALL : CHUNK_PART);
}

// Chunk class when every lane holds the same mask word `w` (before the lane
// shift): the 32 keys (or 16 when one block) of chunk kc.
__device__ inline int uniform_chunk_class(uint64_t w, int kc, bool two_blocks) {
    const uint32_t x = two_blocks ? (uint32_t)(w >> (32 * kc)) : (uint32_t)w & 0xFFFFu;
    const uint32_t full = two_blocks ? 0xFFFFFFFFu : 0xFFFFu;
    return x == 0u ? CHUNK_NONE : (x == full ? CHUNK_ALL : CHUNK_PART);
}

// Row view (the lane owns query row i): constants of the lane.
struct RowLane {
    int i;      // query row
    int i_mod;  // i mod l
    int blk0;   // first column of i's l-block
};
__device__ inline RowLane row_lane(int i, const DivL& dl) {
    const int m = mod_l(dl, i);
    return RowLane{i, m, i - m};
}

// Attended keys j0 + jj (bit jj) of the lane's row, j0 <= i.  j0_mod is
// j0 mod l and sum = summary_bits(j0, l, c) (fixed pattern); both depend on
// the block only.
__device__ inline uint64_t row_mask(const MaskParams& p, const RowLane& x, int j0, int j0_mod, uint64_t sum) {
    const int D = x.i - j0;  // key offset of the diagonal, >= 0
    const uint64_t causal = bit_range(0, D);
    uint64_t a1, a2;
    if (p.pattern == STRIDED) {
        a1 = bit_range(D - p.l, D);
        int m = x.i_mod - j0_mod;  // D mod l
        m += m < 0 ? p.l : 0;
        a2 = periodic_from(p.period_bits, m);
    } else {
        a1 = bit_range(x.blk0 - j0, D);
        a2 = sum;
    }
    const uint64_t m = p.part == PART_A1 ? a1 : (p.part == PART_A2 ? a2 : (a1 | a2));
    return m & causal;
}

// Blocks away from the diagonal.  When every key of a block lies before the
// A1 part of every row of the block (the band of l + 1 keys for strided, the
// row's own l-block for fixed), only A2 can hold there: a period of l along
// the row (strided) or the summary columns (fixed), and causality holds
// everywhere.  Such "far" blocks are most of a long sequence's blocks and get
// these short forms; the general forms above handle the rest.
//   row view, block rows from i0, keys from j0 (B wide):
//     strided: j0 + B - 1 < i0 - l;  fixed: j0 + B - 1 < l floor(i0 / l)
//   column view, block keys up to j1 = j0 + B - 1, rows from i0:
//     strided: i0 > j1 + l;          fixed: i0 > l floor(j1 / l) + l - 1
__device__ inline bool far_block(int pattern, const DivL& dl, int i0, int j0, int B) {
    const int j1 = j0 + B - 1;
    if (pattern == STRIDED) return j1 < i0 - dl.l;
    return j1 < i0 - mod_l(dl, i0);
}

// The steps of a walk along one block row: a step is one present block, or,
// with PAIRS (fixed pattern, B = 64), two consecutive blocks whose attended
// keys, the same for every row, are exactly one half of each (the upper 32
// or the lower 32), computed together as one unmasked block made of the two
// halves.  When c = 32, l is a multiple of 64 and the summary window starts
// at a multiple of 32, every present block away from the diagonal is such a
// block (only one block of an l-block holds summary keys, exactly one half of
// it), and the blocks away from the diagonal are those below far_end, the
// first block of the row's l-block: so one compare per entry decides.
// RowStep::a < 0: the row is done; RowStep::b < 0: block a alone.  Entries are
// read with scalar loads.
struct RowStep {
    int a, b;
};
template <bool PAIRS>
struct RowStepper {
    const int32_t* col_idx;
    int e, e1;    // next entry, end of the row
    int far_end;  // pairs are formed below this key block; 0: no pairs
    bool dense;   // no layout: entry e is key block e
    __device__ static int pair_bound(const MaskParams& p, const DivL& dl, int i0) {
        if (p.pattern != FIXED || p.part == PART_A1 || p.c != 32 || p.l % 64 != 0 || p.w % 32 != 0) return 0;
        return (i0 - mod_l(dl, i0)) / 64;
    }
    __device__ RowStep next() {
        RowStep s{-1, -1};
        if (e >= e1) return s;
        s.a = dense ? e : __builtin_amdgcn_readfirstlane(col_idx[e]);
        ++e;
        if constexpr (PAIRS) {
            if (e < e1) {
                const int kb = __builtin_amdgcn_readfirstlane(col_idx[e]);  // entries ascend: kb > s.a
                if (kb < far_end) {
                    s.b = kb;
                    ++e;
                }
            }
        }
        return s;
    }
};

__device__ inline uint64_t row_mask_far(const MaskParams& p, const RowLane& x, int j0_mod, uint64_t sum) {
    if (p.part == PART_A1) return 0ull;
    if (p.pattern == STRIDED) {
        int m = x.i_mod - j0_mod;  // (i - j0) mod l
        m += m < 0 ? p.l : 0;
        return periodic_from(p.period_bits, m);
    }
    return sum;
}

// Column view (the lane owns key column j): constants of the lane.
struct ColLane {
    int j;         // key column
    int j_mod;     // j mod l
    int blk0;      // first row of j's l-block
    bool summary;  // fixed pattern: w <= j mod l < w + c
};
__device__ inline ColLane col_lane(int j, const DivL& dl, int c, int w) {
    const int m = mod_l(dl, j);
    return ColLane{j, m, j - m, m >= w && m < w + c};
}

// Attended queries i0 + ii (bit ii) of the lane's column; i0_mod = i0 mod l.
__device__ inline uint64_t col_mask(const MaskParams& p, const ColLane& y, int i0, int i0_mod) {
    const int D = y.j - i0;  // query offset of the diagonal (may be negative)
    const uint64_t causal = bit_range(D, 63);
    uint64_t a1, a2;
    if (p.pattern == STRIDED) {
        a1 = bit_range(D, D + p.l);
        int m = y.j_mod - i0_mod;  // D mod l, non-negative
        m += m < 0 ? p.l : 0;
        a2 = periodic_from(p.period_bits, m);
    } else {
        a1 = bit_range(y.blk0 - i0, y.blk0 + p.l - 1 - i0);
        a2 = (p.pattern == FIXED && y.summary) ? ~0ull : 0ull;
    }
    const uint64_t m = p.part == PART_A1 ? a1 : (p.part == PART_A2 ? a2 : (a1 | a2));
    return m & causal;
}

// Far block in the column view (see far_block; the same condition, read for
// the keys): only A2 holds, periodic in the row (strided) or the whole
// column when the key is a summary column (fixed).
__device__ inline uint64_t col_mask_far(const MaskParams& p, const ColLane& y, int i0_mod) {
    if (p.part == PART_A1) return 0ull;
    if (p.pattern == STRIDED) {
        int m = y.j_mod - i0_mod;  // (j - i0) mod l
        m += m < 0 ? p.l : 0;
        return periodic_from(p.period_bits, m);
    }
    return y.summary ? ~0ull : 0ull;
}

// All ones when bit pos (0..63, a constant after unrolling) of bits is set, else 0.
__device__ inline int32_t bit_lane_mask(uint64_t bits, int pos) {
    const uint32_t half = pos < 32 ? (uint32_t)bits : (uint32_t)(bits >> 32);
    return __builtin_amdgcn_sbfe((int32_t)half, (uint32_t)(pos & 31), 1u);
}

// x where the mask is all ones, -inf where it is zero (one bitfield select).
__device__ inline float select_or_neg_inf(int32_t m, float x) {
    return __int_as_float((m & __float_as_int(x)) | (~m & (int32_t)0xff800000));
}

// x where the mask is all ones, +0 where it is zero.
__device__ inline float select_or_zero(int32_t m, float x) { return __int_as_float(m & __float_as_int(x)); }

inline uint64_t host_period_bits(int64_t l) {
    uint64_t bits = 0ull;
    for (int64_t k = 0; k < 64; k += l) bits |= 1ull << k;
    return bits;
}

// Summary positions p < 128 with w <= p mod l < w + c, as two words (fixed,
// l <= 64): the runs w + k l .. w + k l + c - 1.
__host__ __device__ inline void summary_words(int64_t l, int64_t c, int64_t w, uint64_t* lo, uint64_t* hi) {
    uint64_t a = 0ull, b = 0ull;
    if (l <= 64 && c >= 1) {
        for (int64_t s = w; s < 128; s += l) {
            const int64_t e = s + c - 1 < 127 ? s + c - 1 : 127;
            if (s < 64) a |= (~0ull << s) & (~0ull >> (63 - (e < 63 ? e : 63)));
            if (e >= 64) b |= (~0ull << (s > 64 ? s - 64 : 0)) & (~0ull >> (63 - (e - 64)));
        }
    }
    *lo = a;
    *hi = b;
}

}  // namespace sa
