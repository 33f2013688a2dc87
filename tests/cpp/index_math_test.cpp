// Host test of the clustering kernels' cell-index arithmetic
// (cell_coord_clamped): every value maps into [0, ncoord - 1], exactly
// floor((v - v0) / side) when that lies in range, for the cell side 1 that
// an eps of at most 2 quanta gives and for other sides; values below the
// grid origin never give a negative index.
#include <cstdint>
#include <cstdio>
#include <cstdlib>

#include "cluster_common.h"

static int failures = 0;

static void check(int32_t v, int32_t v0, int32_t side, int32_t ncoord) {
    const int32_t got = flock::cl::cell_coord_clamped(v, v0, side, ncoord);
    int64_t want = ((int64_t)v - v0) / side;  // v >= v0 here: truncation is the floor
    if (v < v0) want = ncoord - 1;            // unsigned wrap: the last cell
    if (want > ncoord - 1) want = ncoord - 1;
    if (got != want || got < 0 || got >= ncoord) {
        if (failures++ < 10)
            std::printf("v=%d v0=%d side=%d n=%d: got %d want %lld\n", v, v0, side, ncoord, got, (long long)want);
    }
}

int main() {
    uint64_t s = 88172645463325252ull;
    auto rnd = [&s]() { s ^= s << 13; s ^= s >> 7; s ^= s << 17; return s; };
    const int32_t sides[] = {1, 2, 3, 7, 452, 678, 23170};
    for (int32_t side : sides) {
        for (int t = 0; t < 200000; ++t) {
            const int32_t v0 = (int32_t)(rnd() % (1u << 24));
            const int32_t ext = (int32_t)(rnd() % (1u << 24));
            const int32_t ncoord = (int32_t)(ext / side + 1);
            int32_t v = (int32_t)((uint32_t)v0 + (uint32_t)(rnd() % ((uint64_t)ext + 1)));
            if (t % 7 == 0) v = v0 - 1 - (int32_t)(rnd() % 1000);        // below the origin
            if (t % 11 == 0) v = v0 + ext + 1 + (int32_t)(rnd() % 1000);  // past the far edge
            if (v < 0 || v >= (1 << 24)) continue;
            check(v, v0, side, ncoord);
        }
        check(0, 0, side, 1);
        check((1 << 24) - 1, 0, side, (int32_t)(((1 << 24) - 1) / side + 1));
    }
    if (failures) {
        std::printf("%d failures\n", failures);
        return 1;
    }
    std::printf("index math ok\n");
    return 0;
}
