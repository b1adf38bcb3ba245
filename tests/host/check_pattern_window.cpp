// Host check of the library's closed forms for the fixed pattern with its
// summary window at w .. w + c - 1 of every l-block (w = l - (s + 1) c for
// summary subblock s, Sec. 4.3): each against a brute-force walk over the
// positions, and the head / layout / subblock maps against each other.
#include <cstdio>

#include "sa_mask.h"
#include "sa_pattern.h"

static bool summary(long long j, int l, int c, int w) { return j % l >= w && j % l < w + c; }

static bool attended_ref(int part, int l, int c, int w, long long i, long long j) {
    if (j > i) return false;
    const bool a1 = i / l == j / l, a2 = summary(j, l, c, w);
    return part == 0 ? a1 : (part == 1 ? a2 : (a1 || a2));
}

#define FAIL(...)                 \
    do {                          \
        std::printf(__VA_ARGS__); \
        return 1;                 \
    } while (0)

int main() {
    long long checked = 0;
    const int ls[] = {1, 3, 8, 12, 16, 40, 64, 96, 128, 200};
    for (int l : ls)
        for (int c = 1; c <= l; c += (l > 16 ? l / 8 : 1))
            for (int s = 0; s < l / c; ++s) {
                const int w = (int)sa::summary_start(l, c, s);
                if (w < 0 || w + c > l) FAIL("window out of the block l=%d c=%d s=%d\n", l, c, s);
                sa::Pattern p{sa::FIXED, sa::PART_A2, l, c, w};
                const sa::DivL dl = sa::make_divl(l);
                long long upto = 0;
                for (long long x = 0; x < 4 * l + 70; ++x) {
                    long long first = x;
                    while (!summary(first, l, c, w)) ++first;
                    if (sa::first_summary_at_or_after(x, l, c, w) != first)
                        FAIL("first_summary l=%d c=%d w=%d x=%lld\n", l, c, w, x);
                    upto += summary(x, l, c, w);
                    if (sa::summary_upto(x, l, c, w) != upto) FAIL("summary_upto l=%d c=%d w=%d x=%lld\n", l, c, w, x);
                }
                // summary words (l <= 64): bit p of the 128 positions
                if (l <= 64) {
                    uint64_t lo, hi;
                    sa::summary_words(l, c, w, &lo, &hi);
                    for (int q = 0; q < 128; ++q) {
                        const bool bit = ((q < 64 ? lo >> q : hi >> (q - 64)) & 1ull) != 0;
                        if (bit != summary(q, l, c, w)) FAIL("summary_words l=%d c=%d w=%d p=%d\n", l, c, w, q);
                    }
                }
                // blocks: presence, fullness, counts, element predicate
                for (int B : {4, 16, 64}) {
                    const int nq = (3 * l + 2 * B) / B;
                    for (int part = 0; part < 3; ++part) {
                        p.part = part;
                        for (int qb = 0; qb < nq; ++qb)
                            for (int kb = 0; kb <= qb; ++kb) {
                                const long long r0 = (long long)qb * B, r1 = r0 + B - 1, c0 = (long long)kb * B,
                                                c1 = c0 + B - 1;
                                long long pairs = 0;
                                for (long long i = r0; i <= r1; ++i) {
                                    long long row = 0;
                                    for (long long j = c0; j <= c1; ++j) {
                                        const bool ref = attended_ref(part, l, c, w, i, j);
                                        if (sa::attended(sa::FIXED, part, l, c, w, (int)i, (int)j) != ref)
                                            FAIL("attended l=%d c=%d w=%d i=%lld j=%lld\n", l, c, w, i, j);
                                        row += ref;
                                    }
                                    if (sa::attended_in_range(p, i, c0, c1) != row)
                                        FAIL("attended_in_range l=%d c=%d w=%d part=%d i=%lld\n", l, c, w, part, i);
                                    pairs += row;
                                }
                                if (sa::block_present(p, r0, r1, c0, c1) != (pairs > 0))
                                    FAIL("block_present l=%d c=%d w=%d part=%d B=%d qb=%d kb=%d\n", l, c, w, part, B,
                                         qb, kb);
                                const bool full = pairs == (long long)B * B;
                                const bool f64 = sa::block_full(sa::FIXED, part, l, c, w, r0, r1, c0, c1);
                                const bool f32 = sa::block_full32(sa::FIXED, part, dl, c, w, (int)r0, (int)r1, (int)c0,
                                                                  (int)c1);
                                // exact except fixed merged, where it may miss a full block
                                if (f64 != f32 || (f64 && !full) || (part != 2 && f64 != full))
                                    FAIL("block_full l=%d c=%d w=%d part=%d B=%d qb=%d kb=%d\n", l, c, w, part, B, qb,
                                         kb);
                                ++checked;
                            }
                    }
                }
            }
    // head -> layout -> subblock maps
    for (int mode = 0; mode < 4; ++mode)
        for (int sub : {0, 1, 3, 4, 64}) {
            const int n_layouts = sa::layout_count(mode, sub);
            for (int h = 0; h < 300; ++h) {
                const int g = sa::layout_of_head(mode, sub, h);
                if (g < 0 || g >= n_layouts) FAIL("layout range mode=%d sub=%d h=%d\n", mode, sub, h);
                if (sa::part_of_layout(mode, g) != sa::part_of_head(mode, h))
                    FAIL("layout part mode=%d sub=%d h=%d\n", mode, sub, h);
                if (sa::part_of_head(mode, h) != sa::PART_A1 &&
                    sa::subblock_of_layout(mode, sub, g) != sa::subblock_of_head(sub, h))
                    FAIL("layout subblock mode=%d sub=%d h=%d\n", mode, sub, h);
            }
        }
    std::printf("ok %lld\n", checked);
    return 0;
}
