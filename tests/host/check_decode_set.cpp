// Host check of DecodeSet (the index space over S_pos that the decoding kernel
// walks) against the sets written out from their definitions (Sec. 4.3):
// every position of S_pos exactly once, and nothing else.
#include <cstdio>
#include <vector>

#include "sa_pattern.h"

// Fixed pattern: the summary columns are the positions w .. w + c - 1 of each
// l-block (w = l - c, or l - (s + 1) c for summary subblock s).
static bool in_set(int pattern, int part, int l, int c, int w, int i, int j) {
    if (j < 0 || j > i) return false;
    bool a1, a2;
    if (pattern == 0) {  // strided
        a1 = i - j <= l;
        a2 = (i - j) % l == 0;
    } else {  // fixed
        a1 = i / l == j / l;
        a2 = j % l >= w && j % l < w + c;
    }
    return part == 0 ? a1 : (part == 1 ? a2 : (a1 || a2));
}

int main() {
    long long checked = 0;
    const int ls[] = {1, 2, 3, 5, 8, 16, 31, 64, 100, 128};
    for (int pattern = 0; pattern < 2; ++pattern)
        for (int part = 0; part < 3; ++part)
            for (int l : ls)
                for (int c = (pattern == 0 ? 0 : 1); c <= (pattern == 0 ? 0 : l); c += (l > 8 ? (l + 3) / 4 : 1)) {
                    const sa::DivL dc = sa::make_divl(c > 0 ? c : 1);
                    const int subblocks = pattern == 0 ? 1 : l / c;
                    for (int s = 0; s < subblocks; s += (subblocks > 6 ? subblocks / 3 : 1))
                    for (int pos = 0; pos < 700; ++pos) {
                        const int w = pattern == 0 ? l : (int)sa::summary_start(l, c, s);
                        const sa::DecodeSet S(pattern, part, pos, l, c, w, dc);
                        std::vector<char> seen(pos + 1, 0);
                        for (long long t = 0; t < S.count; ++t) {
                            const int j = S.at(t);
                            if (j < 0 || j > pos || seen[j] || !in_set(pattern, part, l, c, w, pos, j)) {
                                std::printf("bad key pattern=%d part=%d l=%d c=%d w=%d pos=%d t=%lld j=%d\n", pattern,
                                            part, l, c, w, pos, t, j);
                                return 1;
                            }
                            seen[j] = 1;
                        }
                        for (int j = 0; j <= pos; ++j)
                            if (in_set(pattern, part, l, c, w, pos, j) && !seen[j]) {
                                std::printf("missing pattern=%d part=%d l=%d c=%d w=%d pos=%d j=%d\n", pattern, part, l,
                                            c, w, pos, j);
                                return 1;
                            }
                        ++checked;
                    }
                }
    // a position near the top of the range: counts only (closed forms)
    const sa::DecodeSet big(1, 2, 2147483000, 256, 32, 224, sa::make_divl(32));
    if (big.count != (2147483000 % 256) + 1 + (long long)(2147483000 / 256) * 32) {
        std::printf("bad count at large pos\n");
        return 1;
    }
    // A1 from position 0 up to pos = 2^31 - 1 holds 2^31 positions
    const sa::DecodeSet edge(0, 0, 2147483647, 2147483647, 0, 2147483647, sa::make_divl(1));
    if (edge.count != 2147483648ll || edge.at(2147483647ll) != 2147483647) {
        std::printf("bad count at the top of the range\n");
        return 1;
    }
    std::printf("ok %lld\n", checked);
    return 0;
}
