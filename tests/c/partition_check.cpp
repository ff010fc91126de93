// CPU check of the resident schedule's tile division (csrc/fc_partition.h),
// built with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_partition_cpu.py.  For many random plans it checks what the
// kernels rely on: the table covers [0, ntiles) once, in order, round by
// round; equal ranges differ by at most one tile; weighted and balanced
// ranges keep every block within the LDS cap and follow the weights.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "fc_partition.h"

static int failures = 0;
#define CHECK(c, ...)                                   \
    do {                                                \
        if (!(c)) {                                     \
            if (failures++ < 20) {                      \
                std::fprintf(stderr, __VA_ARGS__);      \
                std::fprintf(stderr, " [%s]\n", #c);    \
            }                                           \
        }                                               \
    } while (0)

// table shape, coverage and round boundaries; returns the largest range
static int check_table(const std::vector<int>& t, int ntiles, int rounds, int grid) {
    CHECK(t.size() == static_cast<size_t>(grid) * rounds + 1, "size %zu", t.size());
    if (t.size() != static_cast<size_t>(grid) * rounds + 1) return 0;
    CHECK(t.front() == 0 && t.back() == ntiles, "ends %d %d of %d", t.front(), t.back(), ntiles);
    int most = 0;
    for (size_t i = 0; i + 1 < t.size(); ++i) {
        CHECK(t[i] <= t[i + 1], "not monotone at %zu", i);
        most = std::max(most, t[i + 1] - t[i]);
    }
    for (int r = 0; r <= rounds; ++r) {
        const int want = static_cast<int>(static_cast<uint64_t>(ntiles) * r / rounds);
        CHECK(t[static_cast<size_t>(r) * grid] == want, "round %d starts at %d, not %d", r, t[static_cast<size_t>(r) * grid], want);
    }
    return most;
}

int main() {
    std::mt19937_64 rng(1511);
    int cases = 0, weighted = 0;
    for (int it = 0; it < 4000; ++it) {
        const int grid = 1 + static_cast<int>(rng() % 300);
        const int rounds = 1 + static_cast<int>(rng() % 20);
        const int ntiles = static_cast<int>(rng() % 200000);
        std::vector<int> t;
        fc::equal_ranges(ntiles, rounds, grid, t);
        const int most_eq = check_table(t, ntiles, rounds, grid);
        const int n = grid * rounds;
        const int ceil_eq = (ntiles + n - 1) / n;
        CHECK(most_eq <= ceil_eq, "equal: %d > ceil %d", most_eq, ceil_eq);
        for (size_t i = 0; i + 1 < t.size(); ++i) CHECK(t[i + 1] - t[i] >= ntiles / n, "equal: short range");

        // rates per XCD (b % 8) within +-15%, or per block
        std::vector<double> rel(grid);
        std::uniform_real_distribution<double> u(0.85, 1.15);
        double xr[8];
        for (double& x : xr) x = u(rng);
        const bool per_block = rng() % 4 == 0;
        for (int b = 0; b < grid; ++b) rel[b] = per_block ? u(rng) : xr[b % 8];

        std::vector<int> tw;
        const int most_w = fc::weighted_ranges(ntiles, rounds, grid, rel, tw);
        CHECK(check_table(tw, ntiles, rounds, grid) == most_w, "weighted: reported most differs");
        // shares follow the weights to within two tiles of the exact quotas
        double sum = 0;
        for (double x : rel) sum += x;
        for (int r = 0; r < rounds && grid > 1; ++r) {
            const int lo = tw[static_cast<size_t>(r) * grid], hi = tw[static_cast<size_t>(r + 1) * grid];
            for (int b = 0; b < grid; ++b) {
                const int got = tw[static_cast<size_t>(r) * grid + b + 1] - tw[static_cast<size_t>(r) * grid + b];
                const double want = (hi - lo) * rel[b] / sum;
                CHECK(std::fabs(got - want) <= 2.0, "weighted: block %d got %d, quota %.2f", b, got, want);
            }
        }

        // balanced with an LDS cap between the equal share and 160 slots
        const int cap = std::max(ceil_eq, std::min(160, ceil_eq + static_cast<int>(rng() % 24)));
        std::vector<int> tb;
        const bool follows = fc::balanced_ranges(ntiles, rounds, grid, rel, cap, tb);
        const int most_b = check_table(tb, ntiles, rounds, grid);
        CHECK(most_b <= cap, "balanced: %d tiles > cap %d", most_b, cap);
        if (!follows) CHECK(tb == t, "balanced: fallback is not the equal division");
        weighted += follows;
        ++cases;
    }
    // all weights 1: the weighted division is (within one tile) the equal one
    std::vector<int> t1, te;
    const int most1 = fc::weighted_ranges(27372, 1, 256, std::vector<double>(256, 1.0), t1);
    fc::equal_ranges(27372, 1, 256, te);
    CHECK(most1 <= 107 + 1, "unit weights: %d", most1);
    for (size_t i = 0; i < te.size(); ++i) CHECK(std::abs(t1[i] - te[i]) <= 1, "unit weights differ at %zu", i);
    if (failures) {
        std::fprintf(stderr, "partition_check: %d failures\n", failures);
        return 1;
    }
    std::printf("partition_check: %d random plans, %d rebalanced within the LDS cap, all tables valid\n", cases, weighted);
    return 0;
}
