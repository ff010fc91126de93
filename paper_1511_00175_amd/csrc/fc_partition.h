// Division of the resident schedule's tiles among the blocks of its
// persistent grid: plain host arithmetic, used when a plan is made and by
// fc_plan_balance.  The table holds grid * rounds + 1 tile indices: in round
// r, block b owns tiles [ranges[r * grid + b], ranges[r * grid + b + 1]), and
// round r spans tiles [ntiles * r / rounds, ntiles * (r + 1) / rounds).
#pragma once

#include <algorithm>
#include <cstdint>
#include <vector>

namespace fc {

// Equal division: range i of the grid * rounds ranges is
// [i * ntiles / n, (i + 1) * ntiles / n), n = grid * rounds; at most
// ceil(ntiles / n) tiles each, and round r starts at ntiles * r / rounds.
inline void equal_ranges(int ntiles, int rounds, int grid, std::vector<int>& ranges) {
    const uint64_t n = static_cast<uint64_t>(grid) * rounds;
    ranges.resize(n + 1);
    for (uint64_t i = 0; i <= n; ++i) ranges[i] = static_cast<int>(static_cast<uint64_t>(ntiles) * i / n);
}

// Weighted division: in every round, block b's share of the round's tiles is
// proportional to w[b] (w[b] > 0).  Returns the most tiles any block gets.
inline int weighted_ranges(int ntiles, int rounds, int grid, const std::vector<double>& w, std::vector<int>& ranges) {
    std::vector<double> cum(static_cast<size_t>(grid) + 1, 0.0);
    for (int b = 0; b < grid; ++b) cum[b + 1] = cum[b] + w[b];
    ranges.assign(static_cast<size_t>(grid) * rounds + 1, 0);
    int most = 0;
    for (int r = 0; r < rounds; ++r) {
        const uint64_t lo = static_cast<uint64_t>(ntiles) * r / rounds;
        const uint64_t hi = static_cast<uint64_t>(ntiles) * (r + 1) / rounds;
        const size_t first = static_cast<size_t>(r) * grid;
        ranges[first] = static_cast<int>(lo);
        for (int b = 1; b < grid; ++b) {
            uint64_t x = lo + static_cast<uint64_t>(static_cast<double>(hi - lo) * (cum[b] / cum[grid]));
            x = std::min(hi, std::max<uint64_t>(x, ranges[first + b - 1]));
            ranges[first + b] = static_cast<int>(x);
        }
        ranges[first + grid] = static_cast<int>(hi);  // the next round's first, or the end
        for (int b = 0; b < grid; ++b) most = std::max(most, ranges[first + b + 1] - ranges[first + b]);
    }
    return most;
}

// Shares for per-block relative rates rel[b] (1 = the mean): proportional to
// the rates, with the deviation from equal shares halved (up to six times)
// until no block gets more than `cap` tiles in a round; equal shares when
// even that does not fit.  Returns true when the shares follow the rates.
// Requires cap >= the most tiles of an equal division.
inline bool balanced_ranges(int ntiles, int rounds, int grid, const std::vector<double>& rel, int cap,
                            std::vector<int>& ranges) {
    std::vector<double> w(static_cast<size_t>(grid));
    for (double lam = 1.0; lam >= 1.0 / 64; lam *= 0.5) {
        for (int b = 0; b < grid; ++b) w[b] = 1.0 + lam * (rel[b] - 1.0);
        if (weighted_ranges(ntiles, rounds, grid, w, ranges) <= cap) return true;
    }
    equal_ranges(ntiles, rounds, grid, ranges);
    return false;
}

}  // namespace fc
