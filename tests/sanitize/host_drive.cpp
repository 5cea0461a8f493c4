// Sanitizer driver for the library's host code (test infrastructure): the
// workspace planners, the alias-table builder, the status strings and the
// argument checks of the entry points, none of which touches a GPU.  Built
// with the host side of api.hip and alias.cpp instrumented by
// AddressSanitizer and UndefinedBehaviorSanitizer; run by
// tests/test_sanitize.py.  Exits 0 when every call returns what it should.
#include <stdint.h>
#include <stdio.h>

#include <vector>

#include "huge.h"

static int failures = 0;
#define EXPECT(cond)                                                                   \
    do {                                                                               \
        if (!(cond)) {                                                                 \
            fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                                \
        }                                                                              \
    } while (0)

static huge_config base_config() {
    huge_config c{};
    c.num_nodes = 100000;
    c.dim = 128;
    c.num_neg_per_pos = 5;
    c.max_batch = 4096;
    c.seed = 1;
    c.init_half_width = 0.f;
    c.neg_kind = HUGE_NEG_UNIFORM;
    c.scatter_kind = HUGE_SCATTER_SORTED;
    c.table_dtype = HUGE_DTYPE_F32;
    return c;
}

int main() {
    // workspace planning over the valid ranges and just outside them
    huge_config c = base_config();
    EXPECT(huge_workspace_bytes(&c) > 0);
    EXPECT(huge_workspace_bytes(nullptr) == 0);
    const int64_t nodes[] = {1, 2, 255, 256, 65537, 100000000, 2147483647LL};
    const int32_t dims[] = {4, 8, 12, 128, 260, 520, 1024};
    const int32_t negs[] = {1, 5, 31, 64};
    const int64_t batches[] = {1, 7, 262144, 1 << 22};
    for (int64_t n : nodes)
        for (int32_t d : dims)
            for (int32_t k : negs)
                for (int64_t b : batches)
                    for (int dt = 0; dt < 2; ++dt)
                        for (int sc = 0; sc < 2; ++sc) {
                            huge_config x = base_config();
                            x.num_nodes = n;
                            x.dim = d;
                            x.num_neg_per_pos = k;
                            x.max_batch = b;
                            x.table_dtype = dt;
                            x.scatter_kind = sc;
                            (void)huge_workspace_bytes(&x);
                        }
    huge_config bad = base_config();
    bad.dim = 6;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.num_nodes = 0;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.num_nodes = 2147483648LL;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.num_neg_per_pos = 65;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.max_batch = 0;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.max_batch = INT64_MAX;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.table_dtype = 7;
    EXPECT(huge_workspace_bytes(&bad) == 0);
    bad = base_config();
    bad.neg_kind = 9;
    EXPECT(huge_workspace_bytes(&bad) == 0);

    // walk and evaluation workspaces
    huge_walk_config wc{};
    wc.num_nodes = 1000;
    wc.walks_per_node = 10;
    wc.walk_steps = 40;
    wc.window = 5;  // a seed's walks: 410 nodes, 50 seed pairs
    wc.seed_pairs_only = 1;
    wc.seed = 3;
    EXPECT(huge_walk_workspace_bytes(&wc, 1000) > 0);
    EXPECT(huge_walk_workspace_bytes(&wc, -1) == 0);
    EXPECT(huge_walk_workspace_bytes(nullptr, 10) == 0);
    wc.window = 41;
    EXPECT(huge_walk_workspace_bytes(&wc, 10) == 0);
    wc.window = 10;
    wc.seed_pairs_only = 0;  // 7100 window pairs per seed: above 4096
    EXPECT(huge_walk_workspace_bytes(&wc, 10) == 0);
    (void)huge_eval_workspace_bytes(1000, 100000, 128, 10);
    (void)huge_eval_workspace_bytes(-1, 100000, 128, 10);
    (void)huge_eval_workspace_bytes(1000, 0, 0, 0);

    // alias tables: uniform, skewed with zeros, one bucket, errors
    for (int64_t n : {1, 2, 3, 1000, 65536}) {
        std::vector<double> w((size_t)n);
        for (int64_t j = 0; j < n; ++j) w[(size_t)j] = (j % 7 == 3) ? 0.0 : 1.0 + (double)(j % 13);
        if (n == 1) w[0] = 2.5;
        std::vector<uint32_t> thr((size_t)n);
        std::vector<int32_t> al((size_t)n);
        EXPECT(huge_build_alias(w.data(), n, thr.data(), al.data()) == HUGE_OK);
        for (int64_t j = 0; j < n; ++j) EXPECT(al[(size_t)j] >= 0 && al[(size_t)j] < n);
    }
    {
        double w[3] = {1.0, -1.0, 2.0};
        uint32_t thr[3];
        int32_t al[3];
        EXPECT(huge_build_alias(w, 3, thr, al) == HUGE_ERR_INVALID_ARG);
        double z[3] = {0.0, 0.0, 0.0};
        EXPECT(huge_build_alias(z, 3, thr, al) == HUGE_ERR_INVALID_ARG);
        EXPECT(huge_build_alias(nullptr, 3, thr, al) == HUGE_ERR_INVALID_ARG);
        EXPECT(huge_build_alias(w, 0, thr, al) == HUGE_ERR_INVALID_ARG);
    }

    // status strings and the argument checks that precede any GPU call
    for (int s = -8; s <= 2; ++s) EXPECT(huge_status_string(s) != nullptr);
    huge_destroy(nullptr);
    EXPECT(huge_train_step(nullptr, nullptr, nullptr, nullptr, 1, 0, 0.025f, nullptr, nullptr) ==
           HUGE_ERR_INVALID_ARG);
    EXPECT(huge_prepare_step(nullptr, nullptr, nullptr, nullptr, 1, 0, nullptr) ==
           HUGE_ERR_INVALID_ARG);
    EXPECT(huge_train_prepared(nullptr, 0.025f, nullptr, nullptr) == HUGE_ERR_INVALID_ARG);
    EXPECT(huge_check(nullptr, nullptr) == HUGE_ERR_INVALID_ARG);
    huge_handle* h = nullptr;
    EXPECT(huge_init_tables(nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr,
                            &h) == HUGE_ERR_INVALID_ARG);
    EXPECT(huge_init_tables(&c, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr, &h) ==
           HUGE_ERR_INVALID_ARG);
    EXPECT(h == nullptr);

    if (failures) {
        fprintf(stderr, "%d expectation(s) failed\n", failures);
        return 1;
    }
    printf("host sanitizer drive: ok\n");
    return 0;
}
