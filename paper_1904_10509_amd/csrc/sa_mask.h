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
//   fixed A2          j mod l >= l - c        (c-wide runs at a period of l)
// Elements then test one bit each.
#pragma once

#include <stdint.h>

#include "sa_pattern.h"

namespace sa {

// Bits lo..hi of a 64-bit word (empty when hi < lo); lo, hi may lie outside [0, 63].
__device__ inline uint64_t bit_range(int lo, int hi) {
    lo = lo < 0 ? 0 : lo;
    hi = hi > 63 ? 63 : hi;
    if (hi < lo) return 0ull;
    return (~0ull >> (63 - hi)) & (~0ull << lo);
}

// Bits at positions m, m + l, m + 2l, ... below 64, from `period_bits`
// (bits at 0, l, 2l, ... precomputed for the call).
__device__ inline uint64_t periodic_from(uint64_t period_bits, int m) {
    return m >= 64 ? 0ull : (period_bits << m);
}

// Non-negative remainder.
__device__ inline int mod_pos(int x, int l) {
    int r = x % l;
    return r < 0 ? r + l : r;
}

// Summary columns (j mod l >= l - c) among j0 .. j0 + 63, as bits over j - j0.
__device__ inline uint64_t summary_bits(int j0, int l, int c) {
    const int r0 = j0 % l;
    uint64_t bits = 0ull;
    for (int s = l - c - r0; s <= 63; s += l) bits |= bit_range(s, s + c - 1);
    return bits;
}

struct MaskParams {
    int pattern, part, l, c;
    uint64_t period_bits;  // bits at multiples of l below 64
};

// Row view: attended keys j0 + jj (bit jj) of query row i.  The caller
// guarantees j0 <= i, and passes `sum` = summary_bits(j0, l, c) for the fixed
// pattern (it depends on the block only).
__device__ inline uint64_t row_mask(const MaskParams& p, int i, int j0, uint64_t sum) {
    const int D = i - j0;  // key offset of the diagonal, >= 0
    uint64_t causal = bit_range(0, D);
    uint64_t a1, a2;
    if (p.pattern == STRIDED) {
        a1 = bit_range(D - p.l, D);
        a2 = periodic_from(p.period_bits, D % p.l);
    } else {
        const int bs = i - i % p.l;  // first column of i's l-block
        a1 = bit_range(bs - j0, D);
        a2 = sum;
    }
    uint64_t m = p.part == PART_A1 ? a1 : (p.part == PART_A2 ? a2 : (a1 | a2));
    return m & causal;
}

// Column view: attended queries i0 + ii (bit ii) of key column j.  `summary`
// is whether j is a fixed-pattern summary column.
__device__ inline uint64_t col_mask(const MaskParams& p, int j, int i0, bool summary) {
    const int D = j - i0;  // query offset of the diagonal (may be negative)
    uint64_t causal = bit_range(D, 63);
    uint64_t a1, a2;
    if (p.pattern == STRIDED) {
        a1 = bit_range(D, D + p.l);
        a2 = periodic_from(p.period_bits, mod_pos(D, p.l));
    } else {
        const int bs = j - j % p.l;  // j's l-block
        a1 = bit_range(bs - i0, bs + p.l - 1 - i0);
        a2 = summary ? ~0ull : 0ull;
    }
    uint64_t m = p.part == PART_A1 ? a1 : (p.part == PART_A2 ? a2 : (a1 | a2));
    return m & causal;
}

inline uint64_t host_period_bits(int64_t l) {
    uint64_t bits = 0ull;
    for (int64_t k = 0; k < 64; k += l) bits |= 1ull << k;
    return bits;
}

}  // namespace sa
