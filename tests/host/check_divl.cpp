// Host check of the library's division by the stride l (multiply and shift)
// against exact integer division, over every l up to 70000 and dividends
// that include the ends of the range, multiples of l and their neighbours.
#include <cstdio>
#include <cstdlib>

#include "sa_pattern.h"

int main() {
    long long checked = 0;
    for (int l = 1; l <= 70000; ++l) {
        const sa::DivL d = sa::make_divl(l);
        const int xs[] = {0, 1, l - 1, l, l + 1, 2 * l - 1, 2 * l, 12345, 65535, 65536, 1 << 20,
                          (1 << 30) + 7, 2147483647 - 1, 2147483647, 2147483647 - l, 2147483647 - 2 * l + 1};
        for (int x : xs) {
            if (x < 0) continue;
            const int q = sa::div_l(d, x), r = sa::mod_l(d, x);
            if (q != x / l || r != x % l) {
                std::printf("mismatch l=%d x=%d got %d,%d want %d,%d\n", l, x, q, r, x / l, x % l);
                return 1;
            }
            ++checked;
        }
        for (int k = 0; k < 64; ++k) {  // a spread of multiples of l and neighbours
            const long long base = (long long)l * ((2147483647ll / l) * k / 63);
            for (long long x = base - 1; x <= base + 1; ++x) {
                if (x < 0 || x > 2147483647ll) continue;
                const int q = sa::div_l(d, (int)x);
                if (q != (int)(x / l)) {
                    std::printf("mismatch l=%d x=%lld got %d want %lld\n", l, x, q, x / l);
                    return 1;
                }
                ++checked;
            }
        }
    }
    std::printf("ok %lld\n", checked);
    return 0;
}
