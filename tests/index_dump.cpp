// Prints the library's per-axis window functions (na_index.h, compiled for the
// host) for the problems read from stdin, one line "L k d causal" each: for
// every position x of the axis, in absolute coordinates,
//   start last mask_start inv_lo inv_hi
// of the query at x (window first and last position, the start the kernels'
// mask test uses) and of the key at x (first and last query attending to it).
// tests/test_index_host.py compares them with the oracle.
#include <cstdio>

#include "na_index.h"

int main() {
    int L, k, d, c;
    while (std::scanf("%d %d %d %d", &L, &k, &d, &c) == 4) {
        for (int x = 0; x < L; ++x) {
            const int g = x % d, p = x / d, n = na::group_len(L, d, g);
            const bool cs = c != 0;
            std::printf("%d %d %d %d %d\n", g + d * na::win_start(p, n, k, cs),
                        g + d * na::win_last(p, n, k, cs), g + d * na::mask_start(p, n, k, cs),
                        g + d * na::inv_lo(p, n, k, cs), g + d * na::inv_hi(p, n, k, cs));
        }
    }
    return 0;
}
