// C-ABI host layer of libhuge: argument checks, workspace layout, and the
// launch sequence of each call on the caller's stream.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <new>
#include <vector>

#include "../../include/huge.h"
#include "common.hpp"

using namespace huge;

struct huge_handle {
    huge_config cfg;
    float* S;
    float* T;
    const uint32_t* thr;
    const int32_t* alias;
    uint8_t* ws;
    size_t ws_bytes;
    Layout lay;
    int passes;
    uint32_t epoch;   // counts calls that use the look-back words
    int64_t last_m;   // occurrences of the last sorted step
    // phase timing: (HUGE_PHASES + 1) events per profiled step
    std::vector<hipEvent_t> events;
    int32_t prof_max = 0;
    int32_t prof_used = 0;
};

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool config_ok(const huge_config* c) {
    if (!c) return false;
    if (c->num_nodes < 1 || c->num_nodes > 2147483647LL) return false;
    if (c->dim < 4 || c->dim > kMaxDim || (c->dim % 4) != 0) return false;
    if (c->num_neg_per_pos < 1 || c->num_neg_per_pos > kMaxNeg) return false;
    if (c->max_batch < 1) return false;
    // occurrence indices and sorted positions are 32-bit
    if (c->max_batch > (int64_t)(0x7FFFFFFF / (2 + c->num_neg_per_pos))) return false;
    if (!(c->init_half_width >= 0.0f) || isinf(c->init_half_width)) return false;
    if (c->neg_kind != HUGE_NEG_UNIFORM && c->neg_kind != HUGE_NEG_ALIAS) return false;
    if (c->scatter_kind != HUGE_SCATTER_SORTED && c->scatter_kind != HUGE_SCATTER_ATOMIC)
        return false;
    return true;
}

int key_bits(int64_t N) {
    // keys are in [0, 2N): bits of 2N - 1
    uint64_t top = 2ull * (uint64_t)N - 1ull;
    int b = 0;
    while (top) {
        ++b;
        top >>= 1;
    }
    return b < 1 ? 1 : b;
}

Layout make_layout(const huge_config* c) {
    Layout L;
    const int64_t K = c->num_neg_per_pos;
    const int64_t D = c->dim;
    const int64_t nb = c->max_batch;
    const int64_t M = nb * (2 + K);
    L.max_occ = M;
    L.sort_tiles = (M + kSortTile - 1) / kSortTile;
    L.loss_blocks = (nb + 0) / 1 + 1;  // bounded by one workgroup per positive
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t at = off;
        off = align_up(off + bytes);
        return at;
    };
    L.ctrl = take(sizeof(Control));
    L.hist = take(sizeof(uint32_t) * kMaxPasses * kRadixBins);
    L.lossp = take(sizeof(double) * (size_t)L.loss_blocks);
    L.neg = take(sizeof(int32_t) * (size_t)(nb * K));
    if (c->scatter_kind == HUGE_SCATTER_SORTED) {
        L.keys0 = take(sizeof(uint32_t) * (size_t)M);
        L.keys1 = take(sizeof(uint32_t) * (size_t)M);
        L.vals0 = take(sizeof(uint32_t) * (size_t)M);
        L.vals1 = take(sizeof(uint32_t) * (size_t)M);
        L.info = take(sizeof(int32_t) * (size_t)M);
        L.status = take(sizeof(uint64_t) * (size_t)(L.sort_tiles * kRadixBins));
        const int64_t windows = M / kChunk + 2;
        L.work = take(sizeof(uint4) * (size_t)(windows * kChunk));
        L.wcount = take(sizeof(uint32_t) * (size_t)windows);
        L.longhead = take(sizeof(uint32_t) * (size_t)windows);
        L.wstats = take(sizeof(uint32_t) * (size_t)(windows * 3));
        L.partA = take(sizeof(double) * (size_t)((M / kChunk + 2) * D));
        L.partB = take(sizeof(double) * (size_t)((M / kChunk + 2) * D));
        L.dup = take(sizeof(float) * (size_t)(M * D));
    } else {
        L.gsrc = take(sizeof(float) * (size_t)(nb * D));
        L.coef = take(sizeof(float) * (size_t)(nb * (1 + K)));
    }
    L.total = off;
    return L;
}

template <typename T>
T* at(huge_handle* h, size_t off) {
    return reinterpret_cast<T*>(h->ws + off);
}

TableArgs table_args(huge_handle* h) {
    TableArgs t;
    t.S = h->S;
    t.T = h->T;
    t.N = h->cfg.num_nodes;
    t.D = h->cfg.dim;
    t.K = h->cfg.num_neg_per_pos;
    t.seed = h->cfg.seed;
    t.thr = h->cfg.neg_kind == HUGE_NEG_ALIAS ? h->thr : nullptr;
    t.alias = h->cfg.neg_kind == HUGE_NEG_ALIAS ? h->alias : nullptr;
    return t;
}

#define HIP_TRY(expr)                                   \
    do {                                                \
        if ((expr) != hipSuccess) return HUGE_ERR_HIP;  \
    } while (0)

huge_status create(const huge_config* cfg, float* S, float* T, const uint32_t* thr,
                   const int32_t* alias, void* ws, size_t ws_bytes, huge_handle** out) {
    if (!out) return HUGE_ERR_INVALID_ARG;
    *out = nullptr;
    if (!config_ok(cfg) || !S || !T || !ws) return HUGE_ERR_INVALID_ARG;
    if (cfg->neg_kind == HUGE_NEG_ALIAS && (!thr || !alias)) return HUGE_ERR_INVALID_ARG;
    if (((uintptr_t)S | (uintptr_t)T) % 16 != 0) return HUGE_ERR_INVALID_ARG;
    if ((uintptr_t)ws % kAlign != 0) return HUGE_ERR_INVALID_ARG;
    Layout L = make_layout(cfg);
    if (ws_bytes < L.total) return HUGE_ERR_WORKSPACE;
    huge_handle* h = new (std::nothrow) huge_handle();
    if (!h) return HUGE_ERR_INVALID_ARG;
    h->cfg = *cfg;
    if (h->cfg.init_half_width == 0.0f) h->cfg.init_half_width = 0.5f / (float)cfg->dim;
    h->S = S;
    h->T = T;
    h->thr = thr;
    h->alias = alias;
    h->ws = static_cast<uint8_t*>(ws);
    h->ws_bytes = ws_bytes;
    h->lay = L;
    h->passes = (key_bits(cfg->num_nodes) + kRadixBits - 1) / kRadixBits;
    h->epoch = 0;
    h->last_m = 0;
    *out = h;
    return HUGE_OK;
}

// Zero the control block, and the look-back words, on the stream.
huge_status reset_workspace(huge_handle* h, hipStream_t s) {
    HIP_TRY(hipMemsetAsync(h->ws + h->lay.ctrl, 0, sizeof(Control), s));
    if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED)
        HIP_TRY(launch_clear_status(at<uint64_t>(h, h->lay.status),
                                    h->lay.sort_tiles * kRadixBins, s));
    return HUGE_OK;
}

huge_status check_batch_args(huge_handle* h, const int32_t* src, const int32_t* dst,
                             const int32_t* cc, int64_t n) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    if (n < 0 || n > h->cfg.max_batch) return HUGE_ERR_INVALID_ARG;
    if (n > 0 && (!src || !dst || !cc)) return HUGE_ERR_INVALID_ARG;
    return HUGE_OK;
}

}  // namespace

extern "C" {

size_t huge_workspace_bytes(const huge_config* cfg) {
    if (!config_ok(cfg)) return 0;
    return make_layout(cfg).total;
}

huge_status huge_init_tables(const huge_config* cfg, float* d_S, float* d_T,
                             const uint32_t* d_alias_thr, const int32_t* d_alias,
                             void* d_workspace, size_t ws_bytes, void* stream, huge_handle** out) {
    huge_status st = create(cfg, d_S, d_T, d_alias_thr, d_alias, d_workspace, ws_bytes, out);
    if (st != HUGE_OK) return st;
    huge_handle* h = *out;
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = reset_workspace(h, s);
    if (st == HUGE_OK && launch_init(table_args(h), h->cfg.init_half_width, s) != hipSuccess)
        st = HUGE_ERR_HIP;
    if (st != HUGE_OK) {
        delete h;
        *out = nullptr;
    }
    return st;
}

huge_status huge_attach_tables(const huge_config* cfg, float* d_S, float* d_T,
                               const uint32_t* d_alias_thr, const int32_t* d_alias,
                               void* d_workspace, size_t ws_bytes, huge_handle** out) {
    huge_status st = create(cfg, d_S, d_T, d_alias_thr, d_alias, d_workspace, ws_bytes, out);
    if (st != HUGE_OK) return st;
    st = reset_workspace(*out, nullptr);
    if (st == HUGE_OK && hipStreamSynchronize(nullptr) != hipSuccess) st = HUGE_ERR_HIP;
    if (st != HUGE_OK) {
        delete *out;
        *out = nullptr;
    }
    return st;
}

huge_status huge_train_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                            const int32_t* d_cc, int64_t n, uint64_t first_pos_index, float lr,
                            double* d_loss_sum, void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc, n);
    if (st != HUGE_OK) return st;
    if (!isfinite(lr)) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, L.ctrl);
    uint32_t* hist = at<uint32_t>(h, L.hist);
    double* lossp = at<double>(h, L.lossp);
    int32_t* neg = at<int32_t>(h, L.neg);
    const TableArgs t = table_args(h);
    StepArgs a{d_src, d_dst, d_cc, n, first_pos_index, lr, d_loss_sum};
    const int64_t m = n * (2 + (int64_t)h->cfg.num_neg_per_pos);

    hipEvent_t* ev = nullptr;
    if (h->prof_used < h->prof_max) {
        ev = &h->events[(size_t)h->prof_used * (HUGE_PHASES + 1)];
        h->prof_used += 1;
    }
    auto mark = [&](int k) -> bool { return ev == nullptr || hipEventRecord(ev[k], s) == hipSuccess; };
    if (!mark(0)) return HUGE_ERR_HIP;
    HIP_TRY(launch_begin(ctl, hist, s));
    int64_t blocks = 0;
    if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED) {
        uint32_t* keys[2] = {at<uint32_t>(h, L.keys0), at<uint32_t>(h, L.keys1)};
        uint32_t* vals[2] = {at<uint32_t>(h, L.vals0), at<uint32_t>(h, L.vals1)};
        uint64_t* status = at<uint64_t>(h, L.status);
        HIP_TRY(launch_sample(t, ctl, a, neg, keys[0], hist, h->passes, s));
        if (!mark(1)) return HUGE_ERR_HIP;
        // look-back tags: 8 per call; clear the words when the 30-bit tag wraps
        h->epoch += 1;
        if ((h->epoch & 0x07FFFFFFu) == 0u) {
            HIP_TRY(launch_clear_status(status, L.sort_tiles * kRadixBins, s));
            h->epoch += 1;
        }
        int cur = 0;
        for (int p = 0; p < h->passes; ++p) {
            const uint32_t tag = (h->epoch << 3) | (uint32_t)p;
            HIP_TRY(launch_radix_pass(ctl, keys[cur], p == 0 ? nullptr : vals[cur], keys[cur ^ 1],
                                      vals[cur ^ 1], m, p, hist, status, tag, s));
            cur ^= 1;
        }
        if (!mark(2)) return HUGE_ERR_HIP;
        int32_t* info = at<int32_t>(h, L.info);
        uint4* work = at<uint4>(h, L.work);
        uint32_t* wcount = at<uint32_t>(h, L.wcount);
        uint32_t* longhead = at<uint32_t>(h, L.longhead);
        uint32_t* wstats = at<uint32_t>(h, L.wstats);
        double* partA = at<double>(h, L.partA);
        double* partB = at<double>(h, L.partB);
        float* dup = at<float>(h, L.dup);
        HIP_TRY(launch_mark(ctl, keys[cur], vals[cur], m, t.N, info, work, wcount, longhead,
                            wstats, s));
        if (!mark(3)) return HUGE_ERR_HIP;
        HIP_TRY(launch_fused_step(t, ctl, a, neg, info, dup, lossp, &blocks, s));
        if (!mark(4)) return HUGE_ERR_HIP;
        if (m > 0) {
            HIP_TRY(launch_dup_apply(t, ctl, work, wcount, dup, partA, partB, lr, m, s));
            HIP_TRY(launch_long_combine(t, ctl, longhead, keys[cur], m, partA, partB, lr, s));
        }
        if (!mark(5)) return HUGE_ERR_HIP;
        h->last_m = m;
    } else {
        float* gsrc = at<float>(h, L.gsrc);
        float* coef = at<float>(h, L.coef);
        HIP_TRY(launch_sample(t, ctl, a, neg, nullptr, hist, 0, s));
        if (!mark(1)) return HUGE_ERR_HIP;
        HIP_TRY(launch_atomic_gather(t, ctl, a, neg, gsrc, coef, lossp, &blocks, s));
        if (!mark(2)) return HUGE_ERR_HIP;
        HIP_TRY(launch_atomic_scatter_T(t, ctl, a, neg, coef, s));
        if (!mark(3)) return HUGE_ERR_HIP;
        HIP_TRY(launch_atomic_scatter_S(t, ctl, a, gsrc, s));
        if (!mark(4)) return HUGE_ERR_HIP;
        if (!mark(5)) return HUGE_ERR_HIP;
    }
    if (d_loss_sum) HIP_TRY(launch_loss_final(ctl, lossp, blocks, d_loss_sum, s));
    if (!mark(6)) return HUGE_ERR_HIP;
    return HUGE_OK;
}

huge_status huge_eval_loss(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                           const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                           double* d_loss_sum, void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc, n);
    if (st != HUGE_OK) return st;
    if (!d_loss_sum) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, L.ctrl);
    double* lossp = at<double>(h, L.lossp);
    StepArgs a{d_src, d_dst, d_cc, n, first_pos_index, 0.0f, d_loss_sum};
    HIP_TRY(launch_begin(ctl, at<uint32_t>(h, L.hist), s));
    int64_t blocks = 0;
    HIP_TRY(launch_eval(table_args(h), ctl, a, lossp, &blocks, s));
    HIP_TRY(launch_loss_final(ctl, lossp, blocks, d_loss_sum, s));
    return HUGE_OK;
}

huge_status huge_get_rows(huge_handle* h, int32_t table, const int64_t* d_ids, int64_t n,
                          float* d_out, void* stream) {
    if (!h || (table != 0 && table != 1) || n < 0) return HUGE_ERR_INVALID_ARG;
    if (n == 0) return HUGE_OK;
    if (!d_ids || !d_out) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(launch_get_rows(table_args(h), at<Control>(h, h->lay.ctrl), table, d_ids, n, d_out, s));
    return HUGE_OK;
}

huge_status huge_sample_negatives(huge_handle* h, int64_t n, uint64_t first_pos_index,
                                  int32_t* d_neg_out, void* stream) {
    if (!h || n < 0) return HUGE_ERR_INVALID_ARG;
    if (n == 0) return HUGE_OK;
    if (!d_neg_out) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    StepArgs a{nullptr, nullptr, nullptr, n, first_pos_index, 0.0f, nullptr};
    HIP_TRY(launch_sample(table_args(h), at<Control>(h, h->lay.ctrl), a, d_neg_out, nullptr,
                          nullptr, 0, s));
    return HUGE_OK;
}

huge_status huge_check(huge_handle* h, void* stream) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    Control* ctl = at<Control>(h, h->lay.ctrl);
    uint32_t err = 0;
    HIP_TRY(hipMemcpyAsync(&err, &ctl->error, sizeof(err), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemsetAsync(&ctl->error, 0, sizeof(uint32_t), s));
    HIP_TRY(hipStreamSynchronize(s));
    if (err == kBadId) return HUGE_ERR_ID_OUT_OF_RANGE;
    if (err == kBadCount) return HUGE_ERR_BAD_COUNT;
    if (err != 0) return HUGE_ERR_HIP;
    return HUGE_OK;
}

huge_status huge_step_stats(huge_handle* h, void* stream, int64_t* unique_src,
                            int64_t* unique_ctx, int64_t* dup_occurrences) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    const bool sorted = h->cfg.scatter_kind == HUGE_SCATTER_SORTED;
    int64_t a = -1, b = -1, c = -1;
    if (sorted) {
        hipStream_t s = static_cast<hipStream_t>(stream);
        const int64_t windows = (h->last_m + kChunk - 1) / kChunk;
        std::vector<uint32_t> w((size_t)windows * 3);
        if (windows > 0)
            HIP_TRY(hipMemcpyAsync(w.data(), h->ws + h->lay.wstats, w.size() * sizeof(uint32_t),
                                   hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        a = b = c = 0;
        for (int64_t i = 0; i < windows; ++i) {
            a += w[(size_t)i * 3];
            b += w[(size_t)i * 3 + 1];
            c += w[(size_t)i * 3 + 2];
        }
    }
    if (unique_src) *unique_src = a;
    if (unique_ctx) *unique_ctx = b;
    if (dup_occurrences) *dup_occurrences = c;
    return HUGE_OK;
}

static void release_events(huge_handle* h) {
    for (hipEvent_t e : h->events) (void)hipEventDestroy(e);
    h->events.clear();
    h->prof_max = 0;
    h->prof_used = 0;
}

huge_status huge_profile_begin(huge_handle* h, int32_t max_steps) {
    if (!h || max_steps < 1 || max_steps > 1000000) return HUGE_ERR_INVALID_ARG;
    release_events(h);
    h->events.resize((size_t)max_steps * (HUGE_PHASES + 1), nullptr);
    for (auto& e : h->events) {
        if (hipEventCreate(&e) != hipSuccess) {
            e = nullptr;
            release_events(h);
            return HUGE_ERR_HIP;
        }
    }
    h->prof_max = max_steps;
    h->prof_used = 0;
    return HUGE_OK;
}

huge_status huge_profile_end(huge_handle* h, void* stream, double* phase_ms, int32_t* steps) {
    if (!h || !phase_ms || !steps) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    huge_status st = HUGE_OK;
    if (hipStreamSynchronize(s) != hipSuccess) st = HUGE_ERR_HIP;
    for (int k = 0; k < HUGE_PHASES; ++k) phase_ms[k] = 0.0;
    for (int32_t i = 0; st == HUGE_OK && i < h->prof_used; ++i) {
        hipEvent_t* ev = &h->events[(size_t)i * (HUGE_PHASES + 1)];
        for (int k = 0; k < HUGE_PHASES; ++k) {
            float ms = 0.0f;
            if (hipEventElapsedTime(&ms, ev[k], ev[k + 1]) != hipSuccess) {
                st = HUGE_ERR_HIP;
                break;
            }
            phase_ms[k] += (double)ms;
        }
    }
    *steps = h->prof_used;
    release_events(h);
    return st;
}

void huge_destroy(huge_handle* h) {
    if (!h) return;
    release_events(h);
    delete h;
}

const char* huge_status_string(huge_status st) {
    switch (st) {
        case HUGE_OK: return "ok";
        case HUGE_ERR_INVALID_ARG: return "invalid argument";
        case HUGE_ERR_ID_OUT_OF_RANGE: return "id out of range";
        case HUGE_ERR_BAD_COUNT: return "negative co_count";
        case HUGE_ERR_WORKSPACE: return "workspace too small";
        case HUGE_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

}  // extern "C"
