// huge_build_alias: exact-integer alias table (Walker 1977; Vose 1991) for
// drawing negatives in proportion to caller weights.
//
// Bucket j starts with mass W_j = trunc(w_j * (N * 2^32 / sum w)) in units of
// 2^-32 of a bucket; the residue N * 2^32 - sum W goes to the largest bucket
// (lowest index on ties) so the masses add up exactly.  Buckets below one
// unit of 2^32 ("small") are topped up, in FIFO index order, by the first
// "large" bucket, which keeps the remainder and turns small when it drops
// below 2^32.  Buckets left at the end hold exactly 2^32 and keep themselves.
#include <math.h>
#include <stdint.h>

#include <deque>
#include <vector>

#include "../../include/huge.h"

extern "C" huge_status huge_build_alias(const double* weights, int64_t n, uint32_t* thr_out,
                                        int32_t* alias_out) {
    if (!weights || !thr_out || !alias_out || n < 1 || n > 2147483647LL)
        return HUGE_ERR_INVALID_ARG;
    double sum = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        const double w = weights[j];
        if (!(w >= 0.0) || !isfinite(w)) return HUGE_ERR_INVALID_ARG;
        sum += w;
    }
    if (!(sum > 0.0) || !isfinite(sum)) return HUGE_ERR_INVALID_ARG;

    constexpr uint64_t kUnit = 1ull << 32;
    const double units_per_weight = (double)n * 4294967296.0 / sum;
    std::vector<uint64_t> mass((size_t)n);
    uint64_t total = 0;
    int64_t largest = 0;
    for (int64_t j = 0; j < n; ++j) {
        mass[(size_t)j] = (uint64_t)(weights[j] * units_per_weight);
        total += mass[(size_t)j];
        if (mass[(size_t)j] > mass[(size_t)largest]) largest = j;
    }
    mass[(size_t)largest] += (uint64_t)n * kUnit - total;  // modular: exact signed residue

    std::deque<int64_t> small, large;
    for (int64_t j = 0; j < n; ++j) {
        thr_out[j] = 0xFFFFFFFFu;
        alias_out[j] = (int32_t)j;
        (mass[(size_t)j] < kUnit ? small : large).push_back(j);
    }
    while (!small.empty() && !large.empty()) {
        const int64_t s = small.front();
        small.pop_front();
        const int64_t l = large.front();
        thr_out[s] = (uint32_t)mass[(size_t)s];
        alias_out[s] = (int32_t)l;
        mass[(size_t)l] -= kUnit - mass[(size_t)s];
        if (mass[(size_t)l] < kUnit) {
            large.pop_front();
            small.push_back(l);
        }
    }
    return HUGE_OK;
}
