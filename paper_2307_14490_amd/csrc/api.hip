// C-ABI host layer of libhuge: argument checks, workspace layout, and the
// launch sequence of each call on the caller's stream.
//
// A step has two halves.  Grouping (k_begin, k_sample, the radix passes,
// k_mark) reads only the batch; applying (k_fused_step, the repeated-row
// kernels, the loss) reads and writes the tables.  Two grouping slots let
// the caller group batch t+1 on one stream while batch t is applied on
// another; events recorded here order the two: an apply waits until its
// slot's grouping is complete, a grouping waits until the previous apply
// that used its slot is complete.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <new>
#include <vector>

#include "../../include/huge.h"
#include "common.hpp"

using namespace huge;

namespace {

constexpr int kSlots = 2;
constexpr int kPrepEvents = 4;   // begin, after sampling, after sort, after marking
constexpr int kApplyEvents = 4;  // begin, after fused step, after repeated rows, after loss

struct PendingBatch {
    const int32_t* src = nullptr;
    const int32_t* dst = nullptr;
    const int32_t* cc = nullptr;
    int64_t n = 0;
    uint64_t first_pos = 0;
};

}  // namespace

struct huge_handle {
    huge_config cfg;
    float* S;
    float* T;
    const uint32_t* thr;
    const int32_t* alias;
    uint8_t* ws;
    size_t ws_bytes;
    Layout lay;
    SortPlan plan;  // radix passes and digit width for keys below 2N
    int key_bits;   // bits of 2N - 1
    uint32_t epoch;            // tags the look-back words of each grouping
    int64_t prepared;          // groupings issued
    int64_t applied;           // applies issued
    int last_applied_slot;     // -1 before the first apply
    PendingBatch pending[kSlots];
    hipEvent_t ready[kSlots];  // grouping of the slot complete
    hipEvent_t done[kSlots];   // apply of the slot complete
    // phase timing
    std::vector<hipEvent_t> prep_ev, apply_ev;
    int32_t prof_max = 0, prof_prep = 0, prof_apply = 0;
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
    const bool sorted = c->scatter_kind == HUGE_SCATTER_SORTED;
    L.max_occ = M;
    L.sort_tiles = (M + kSortTile - 1) / kSortTile;
    L.windows = M / kChunk + 2;
    L.loss_blocks = nb + 1;  // at most one workgroup per positive
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t at = off;
        off = align_up(off + bytes);
        return at;
    };
    for (int s = 0; s < kSlots; ++s) {
        SlotLayout& S = L.slot[s];
        S.ctrl = take(sizeof(Control));
        S.hist = take(sizeof(uint32_t) * kMaxPasses * kMaxBins);
        S.neg = take(sizeof(int32_t) * (size_t)(nb * K));
        if (sorted) {
            S.keys0 = take(sizeof(uint32_t) * (size_t)M);
            S.keys1 = take(sizeof(uint32_t) * (size_t)M);
            S.vals0 = take(sizeof(uint32_t) * (size_t)M);
            S.vals1 = take(sizeof(uint32_t) * (size_t)M);
            S.info = take(sizeof(int32_t) * (size_t)M);
            S.status = take(sizeof(uint64_t) * (size_t)(L.sort_tiles * kMaxBins));
            S.bstart = take(sizeof(uint32_t) * kMaxBins);
            S.biglist = take(sizeof(uint32_t) * kMaxBins);
            S.work = take(sizeof(uint4) * (size_t)(L.windows * kChunk));
            S.wcount = take(sizeof(uint32_t) * (size_t)L.windows);
            S.longhead = take(sizeof(uint32_t) * (size_t)L.windows);
            S.wstats = take(sizeof(uint32_t) * (size_t)(L.windows * 3));
        }
    }
    L.eval_ctrl = take(sizeof(Control));
    L.lossp = take(sizeof(double) * (size_t)L.loss_blocks);
    if (sorted) {
        L.partA = take(sizeof(double) * (size_t)(L.windows * D));
        L.partB = take(sizeof(double) * (size_t)(L.windows * D));
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

void release_profile(huge_handle* h) {
    for (hipEvent_t e : h->prep_ev)
        if (e) (void)hipEventDestroy(e);
    for (hipEvent_t e : h->apply_ev)
        if (e) (void)hipEventDestroy(e);
    h->prep_ev.clear();
    h->apply_ev.clear();
    h->prof_max = h->prof_prep = h->prof_apply = 0;
}

void destroy_handle(huge_handle* h) {
    if (!h) return;
    release_profile(h);
    for (int s = 0; s < kSlots; ++s) {
        if (h->ready[s]) (void)hipEventDestroy(h->ready[s]);
        if (h->done[s]) (void)hipEventDestroy(h->done[s]);
    }
    delete h;
}

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
    h->key_bits = key_bits(cfg->num_nodes);
    h->plan = sort_plan(h->key_bits);
    h->epoch = 0;
    h->prepared = h->applied = 0;
    h->last_applied_slot = -1;
    for (int s = 0; s < kSlots; ++s) h->ready[s] = h->done[s] = nullptr;
    for (int s = 0; s < kSlots; ++s) {
        if (hipEventCreateWithFlags(&h->ready[s], hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&h->done[s], hipEventDisableTiming) != hipSuccess) {
            destroy_handle(h);
            return HUGE_ERR_HIP;
        }
    }
    *out = h;
    return HUGE_OK;
}

// Zero the control blocks and the look-back words, on the stream.
huge_status reset_workspace(huge_handle* h, hipStream_t s) {
    for (int k = 0; k < kSlots; ++k) {
        HIP_TRY(hipMemsetAsync(h->ws + h->lay.slot[k].ctrl, 0, sizeof(Control), s));
        if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED) {
            HIP_TRY(launch_clear_status(at<uint64_t>(h, h->lay.slot[k].status),
                                        h->lay.sort_tiles * kMaxBins, s));
            HIP_TRY(launch_fill_i32(at<int32_t>(h, h->lay.slot[k].info), -1, h->lay.max_occ, s));
        }
    }
    HIP_TRY(hipMemsetAsync(h->ws + h->lay.eval_ctrl, 0, sizeof(Control), s));
    return HUGE_OK;
}

huge_status check_batch_args(huge_handle* h, const int32_t* src, const int32_t* dst,
                             const int32_t* cc, int64_t n) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    if (n < 0 || n > h->cfg.max_batch) return HUGE_ERR_INVALID_ARG;
    if (n > 0 && (!src || !dst || !cc)) return HUGE_ERR_INVALID_ARG;
    return HUGE_OK;
}

// Grouping of one batch into the next slot (launches only; arguments checked).
huge_status group_batch(huge_handle* h, const int32_t* src, const int32_t* dst,
                        const int32_t* cc, int64_t n, uint64_t first_pos, hipStream_t s) {
    const int slot = (int)(h->prepared % kSlots);
    const SlotLayout& SL = h->lay.slot[slot];
    Control* ctl = at<Control>(h, SL.ctrl);
    uint32_t* hist = at<uint32_t>(h, SL.hist);
    int32_t* neg = at<int32_t>(h, SL.neg);
    const TableArgs t = table_args(h);
    const StepArgs a{src, dst, cc, n, first_pos, 0.0f, nullptr};
    const int64_t m = n * (2 + (int64_t)h->cfg.num_neg_per_pos);

    hipEvent_t* ev = nullptr;
    if (h->prof_prep < h->prof_max) ev = &h->prep_ev[(size_t)h->prof_prep++ * kPrepEvents];
    auto mark = [&](int k) -> bool {
        return ev == nullptr || hipEventRecord(ev[k], s) == hipSuccess;
    };

    // the slot's previous apply must be complete before its buffers change
    HIP_TRY(hipStreamWaitEvent(s, h->done[slot], 0));
    if (!mark(0)) return HUGE_ERR_HIP;
    HIP_TRY(launch_begin(ctl, hist, s));
    if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED) {
        uint32_t* keys[2] = {at<uint32_t>(h, SL.keys0), at<uint32_t>(h, SL.keys1)};
        uint32_t* vals[2] = {at<uint32_t>(h, SL.vals0), at<uint32_t>(h, SL.vals1)};
        uint64_t* status = at<uint64_t>(h, SL.status);
        HIP_TRY(launch_sample(t, ctl, a, neg, keys[0], at<int32_t>(h, SL.info), hist, h->plan,
                              s));
        if (!mark(1)) return HUGE_ERR_HIP;
        // look-back tags: 8 per grouping; the words are cleared when the
        // 30-bit tag wraps
        h->epoch += 1;
        if ((h->epoch & 0x07FFFFFFu) == 0u) {
            for (int k = 0; k < kSlots; ++k)
                HIP_TRY(launch_clear_status(at<uint64_t>(h, h->lay.slot[k].status),
                                            h->lay.sort_tiles * kMaxBins, s));
            h->epoch += 1;
        }
        // First pass: buckets by the lowest digit.  Then each bucket is
        // sorted in LDS into the buffer the full sort would end in; the later
        // passes run only if a bucket was too large for that (ctl->overflow).
        const int fin = h->plan.passes & 1;
        uint32_t* bstart = at<uint32_t>(h, SL.bstart);
        HIP_TRY(launch_radix_pass(ctl, keys[0], nullptr, keys[1], vals[1], m, 0, h->plan.bits,
                                  hist, status, h->epoch << 3, nullptr, bstart, s));
        if (h->plan.passes > 1) {
            HIP_TRY(launch_bucket_sort(ctl, keys[1], vals[1], keys[fin], vals[fin], m,
                                       h->plan.bits, h->key_bits, hist, bstart,
                                       at<uint32_t>(h, SL.biglist), s));
            int cur = 1;
            for (int p = 1; p < h->plan.passes; ++p) {
                const uint32_t tag = (h->epoch << 3) | (uint32_t)p;
                HIP_TRY(launch_radix_pass(ctl, keys[cur], vals[cur], keys[cur ^ 1], vals[cur ^ 1],
                                          m, p, h->plan.bits, hist, status, tag, &ctl->overflow,
                                          nullptr, s));
                cur ^= 1;
            }
        }
        const int cur = fin;
        if (!mark(2)) return HUGE_ERR_HIP;
        HIP_TRY(launch_mark(ctl, keys[cur], vals[cur], m, t.N, at<int32_t>(h, SL.info),
                            at<uint4>(h, SL.work), at<uint32_t>(h, SL.wcount),
                            at<uint32_t>(h, SL.longhead), at<uint32_t>(h, SL.wstats), s));
        if (!mark(3)) return HUGE_ERR_HIP;
    } else {
        HIP_TRY(launch_sample(t, ctl, a, neg, nullptr, nullptr, hist, h->plan, s));
        if (!mark(1) || !mark(2) || !mark(3)) return HUGE_ERR_HIP;
    }
    HIP_TRY(hipEventRecord(h->ready[slot], s));
    h->pending[slot] = PendingBatch{src, dst, cc, n, first_pos};
    h->prepared += 1;
    return HUGE_OK;
}

// Apply the oldest grouped batch (launches only).
huge_status apply_batch(huge_handle* h, float lr, double* loss_out, hipStream_t s) {
    const int slot = (int)(h->applied % kSlots);
    const SlotLayout& SL = h->lay.slot[slot];
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, SL.ctrl);
    const PendingBatch& b = h->pending[slot];
    const TableArgs t = table_args(h);
    const StepArgs a{b.src, b.dst, b.cc, b.n, b.first_pos, lr, loss_out};
    const int64_t m = b.n * (2 + (int64_t)h->cfg.num_neg_per_pos);
    int32_t* neg = at<int32_t>(h, SL.neg);
    double* lossp = at<double>(h, L.lossp);

    hipEvent_t* ev = nullptr;
    if (h->prof_apply < h->prof_max) ev = &h->apply_ev[(size_t)h->prof_apply++ * kApplyEvents];
    auto mark = [&](int k) -> bool {
        return ev == nullptr || hipEventRecord(ev[k], s) == hipSuccess;
    };

    HIP_TRY(hipStreamWaitEvent(s, h->ready[slot], 0));
    // applies write the tables and share the apply regions: one at a time
    if (h->last_applied_slot >= 0)
        HIP_TRY(hipStreamWaitEvent(s, h->done[h->last_applied_slot], 0));
    if (!mark(0)) return HUGE_ERR_HIP;
    int64_t blocks = 0;
    if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED) {
        const uint32_t* keys_sorted = at<uint32_t>(h, (h->plan.passes & 1) ? SL.keys1 : SL.keys0);
        double* partA = at<double>(h, L.partA);
        double* partB = at<double>(h, L.partB);
        float* dup = at<float>(h, L.dup);
        HIP_TRY(launch_fused_step(t, ctl, a, neg, at<int32_t>(h, SL.info), dup, lossp, &blocks,
                                  s));
        if (!mark(1)) return HUGE_ERR_HIP;
        if (m > 0) {
            HIP_TRY(launch_dup_apply(t, ctl, at<uint4>(h, SL.work), at<uint32_t>(h, SL.wcount),
                                     dup, partA, partB, lr, m, s));
            HIP_TRY(launch_long_combine(t, ctl, at<uint32_t>(h, SL.longhead), keys_sorted, m,
                                        partA, partB, lr, s));
        }
        if (!mark(2)) return HUGE_ERR_HIP;
    } else {
        float* gsrc = at<float>(h, L.gsrc);
        float* coef = at<float>(h, L.coef);
        HIP_TRY(launch_atomic_gather(t, ctl, a, neg, gsrc, coef, lossp, &blocks, s));
        if (!mark(1)) return HUGE_ERR_HIP;
        HIP_TRY(launch_atomic_scatter_T(t, ctl, a, neg, coef, s));
        HIP_TRY(launch_atomic_scatter_S(t, ctl, a, gsrc, s));
        if (!mark(2)) return HUGE_ERR_HIP;
    }
    if (loss_out) HIP_TRY(launch_loss_final(ctl, lossp, blocks, loss_out, s));
    if (!mark(3)) return HUGE_ERR_HIP;
    HIP_TRY(hipEventRecord(h->done[slot], s));
    h->last_applied_slot = slot;
    h->applied += 1;
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
        destroy_handle(h);
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
        destroy_handle(*out);
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
    if (h->prepared != h->applied) return HUGE_ERR_INVALID_ARG;  // a prepared batch is pending
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = group_batch(h, d_src, d_dst, d_cc, n, first_pos_index, s);
    if (st != HUGE_OK) return st;
    return apply_batch(h, lr, d_loss_sum, s);
}

huge_status huge_prepare_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                              const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                              void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc, n);
    if (st != HUGE_OK) return st;
    if (h->prepared - h->applied >= kSlots) return HUGE_ERR_INVALID_ARG;
    return group_batch(h, d_src, d_dst, d_cc, n, first_pos_index,
                       static_cast<hipStream_t>(stream));
}

huge_status huge_train_prepared(huge_handle* h, float lr, double* d_loss_sum, void* stream) {
    if (!h || !isfinite(lr)) return HUGE_ERR_INVALID_ARG;
    if (h->applied >= h->prepared) return HUGE_ERR_INVALID_ARG;  // nothing prepared
    return apply_batch(h, lr, d_loss_sum, static_cast<hipStream_t>(stream));
}

huge_status huge_eval_loss(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                           const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                           double* d_loss_sum, void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc, n);
    if (st != HUGE_OK) return st;
    if (!d_loss_sum) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, L.eval_ctrl);
    // the loss partials are shared with applies: order after the last one
    if (h->last_applied_slot >= 0)
        HIP_TRY(hipStreamWaitEvent(s, h->done[h->last_applied_slot], 0));
    double* lossp = at<double>(h, L.lossp);
    StepArgs a{d_src, d_dst, d_cc, n, first_pos_index, 0.0f, d_loss_sum};
    HIP_TRY(launch_begin(ctl, nullptr, s));
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
    HIP_TRY(launch_get_rows(table_args(h), at<Control>(h, h->lay.eval_ctrl), table, d_ids, n,
                            d_out, s));
    return HUGE_OK;
}

huge_status huge_probe_rows(huge_handle* h, const int32_t* d_src, const int32_t* d_dst, int64_t n,
                            uint64_t first_pos_index, void* stream) {
    if (!h || n < 0 || n > h->cfg.max_batch) return HUGE_ERR_INVALID_ARG;
    if (n == 0) return HUGE_OK;
    if (!d_src || !d_dst) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // the tables are shared with applies: order after the last one
    if (h->last_applied_slot >= 0)
        HIP_TRY(hipStreamWaitEvent(s, h->done[h->last_applied_slot], 0));
    HIP_TRY(launch_probe(table_args(h), at<Control>(h, h->lay.eval_ctrl), d_src, d_dst, n,
                         first_pos_index, s));
    return HUGE_OK;
}

huge_status huge_sample_negatives(huge_handle* h, int64_t n, uint64_t first_pos_index,
                                  int32_t* d_neg_out, void* stream) {
    if (!h || n < 0) return HUGE_ERR_INVALID_ARG;
    if (n == 0) return HUGE_OK;
    if (!d_neg_out) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    StepArgs a{nullptr, nullptr, nullptr, n, first_pos_index, 0.0f, nullptr};
    HIP_TRY(launch_sample(table_args(h), at<Control>(h, h->lay.eval_ctrl), a, d_neg_out, nullptr,
                          nullptr, nullptr, h->plan, s));
    return HUGE_OK;
}

namespace {

// Pairs one walk of steps + 1 nodes contributes at most.
int64_t walk_pairs_per_walk(const huge_walk_config* c) {
    if (c->seed_pairs_only) return c->window;
    const int64_t w = c->window, L = c->walk_steps + 1;
    return 2 * (w * L - w * (w + 1) / 2);
}

bool walk_config_ok(const huge_walk_config* c) {
    if (!c) return false;
    if (c->num_nodes < 1 || c->num_nodes > 2147483647LL) return false;
    if (c->walks_per_node < 1 || c->walks_per_node > kWalkMaxWalks) return false;
    if (c->walk_steps < 1 || c->walk_steps > kWalkMaxSteps) return false;
    if (c->window < 1 || c->window > c->walk_steps || c->window > kWalkMaxWindow) return false;
    if (c->seed_pairs_only != 0 && c->seed_pairs_only != 1) return false;
    if ((int64_t)c->walks_per_node * (c->walk_steps + 1) > kWalkMaxNodes) return false;
    if ((int64_t)c->walks_per_node * walk_pairs_per_walk(c) > kWalkMaxPairs) return false;
    return true;
}

}  // namespace

size_t huge_walk_workspace_bytes(const huge_walk_config* cfg, int64_t num_seeds) {
    if (!walk_config_ok(cfg) || num_seeds < 0) return 0;
    const size_t n = (size_t)(num_seeds > 0 ? num_seeds : 1);
    return align_up(sizeof(uint64_t) * n) + align_up(sizeof(uint32_t) * n);
}

huge_status huge_sample_walks(const huge_walk_config* cfg, const int64_t* d_offsets,
                              const int32_t* d_neighbors, int64_t num_edges, int64_t first_seed,
                              int64_t num_seeds, int32_t* d_src, int32_t* d_dst, int32_t* d_cc,
                              int32_t* d_hist, int64_t capacity, int64_t* d_count,
                              int32_t* d_status, void* d_workspace, size_t ws_bytes,
                              void* stream) {
    if (!walk_config_ok(cfg) || !d_offsets || num_edges < 0 || (num_edges > 0 && !d_neighbors))
        return HUGE_ERR_INVALID_ARG;
    if (first_seed < 0 || num_seeds < 0 || first_seed + num_seeds > cfg->num_nodes)
        return HUGE_ERR_INVALID_ARG;
    if (capacity < 0 || !d_count || !d_status || !d_workspace) return HUGE_ERR_INVALID_ARG;
    if (capacity > 0 && (!d_src || !d_dst || !d_cc)) return HUGE_ERR_INVALID_ARG;
    if ((uintptr_t)d_workspace % kAlign != 0) return HUGE_ERR_INVALID_ARG;
    if (ws_bytes < huge_walk_workspace_bytes(cfg, num_seeds)) return HUGE_ERR_WORKSPACE;
    const size_t n = (size_t)(num_seeds > 0 ? num_seeds : 1);
    uint8_t* ws = static_cast<uint8_t*>(d_workspace);
    uint64_t* offsets = reinterpret_cast<uint64_t*>(ws);
    uint32_t* counts = reinterpret_cast<uint32_t*>(ws + align_up(sizeof(uint64_t) * n));
    WalkArgs A;
    A.off = d_offsets;
    A.nbr = d_neighbors;
    A.num_nodes = cfg->num_nodes;
    A.num_edges = num_edges;
    A.walks = cfg->walks_per_node;
    A.steps = cfg->walk_steps;
    A.window = cfg->window;
    A.seed_only = cfg->seed_pairs_only;
    A.seed = cfg->seed;
    A.first_seed = first_seed;
    A.num_seeds = num_seeds;
    HIP_TRY(launch_walks(A, counts, offsets, d_count, capacity, d_src, d_dst, d_cc, d_hist,
                         d_status, static_cast<hipStream_t>(stream)));
    return HUGE_OK;
}

huge_status huge_check(huge_handle* h, void* stream) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // every grouping and apply issued so far, on any stream
    for (int k = 0; k < kSlots; ++k) {
        HIP_TRY(hipStreamWaitEvent(s, h->ready[k], 0));
        HIP_TRY(hipStreamWaitEvent(s, h->done[k], 0));
    }
    const size_t ctrls[3] = {h->lay.slot[0].ctrl, h->lay.slot[1].ctrl, h->lay.eval_ctrl};
    uint32_t err[3] = {0, 0, 0};
    for (int k = 0; k < 3; ++k) {
        Control* c = at<Control>(h, ctrls[k]);
        HIP_TRY(hipMemcpyAsync(&err[k], &c->error, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemsetAsync(&c->error, 0, sizeof(uint32_t), s));
    }
    HIP_TRY(hipStreamSynchronize(s));
    uint32_t first = 0;
    for (int k = 0; k < 3; ++k)
        if (!first) first = err[k];
    if (first == kBadId) return HUGE_ERR_ID_OUT_OF_RANGE;
    if (first == kBadCount) return HUGE_ERR_BAD_COUNT;
    if (first != 0) return HUGE_ERR_HIP;
    return HUGE_OK;
}

huge_status huge_step_stats(huge_handle* h, void* stream, int64_t* unique_src,
                            int64_t* unique_ctx, int64_t* dup_occurrences) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    const bool sorted = h->cfg.scatter_kind == HUGE_SCATTER_SORTED;
    int64_t a = -1, b = -1, c = -1;
    if (sorted && h->last_applied_slot >= 0) {
        const int slot = h->last_applied_slot;
        hipStream_t s = static_cast<hipStream_t>(stream);
        HIP_TRY(hipStreamWaitEvent(s, h->done[slot], 0));
        const int64_t m = h->pending[slot].n * (2 + (int64_t)h->cfg.num_neg_per_pos);
        const int64_t windows = (m + kChunk - 1) / kChunk;
        std::vector<uint32_t> w((size_t)windows * 3);
        if (windows > 0)
            HIP_TRY(hipMemcpyAsync(w.data(), h->ws + h->lay.slot[slot].wstats,
                                   w.size() * sizeof(uint32_t), hipMemcpyDeviceToHost, s));
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

huge_status huge_profile_begin(huge_handle* h, int32_t max_steps) {
    if (!h || max_steps < 1 || max_steps > 1000000) return HUGE_ERR_INVALID_ARG;
    release_profile(h);
    h->prep_ev.assign((size_t)max_steps * kPrepEvents, nullptr);
    h->apply_ev.assign((size_t)max_steps * kApplyEvents, nullptr);
    for (std::vector<hipEvent_t>* v : {&h->prep_ev, &h->apply_ev}) {
        for (hipEvent_t& e : *v) {
            if (hipEventCreate(&e) != hipSuccess) {
                e = nullptr;
                release_profile(h);
                return HUGE_ERR_HIP;
            }
        }
    }
    h->prof_max = max_steps;
    return HUGE_OK;
}

huge_status huge_profile_end(huge_handle* h, void* stream, double* phase_ms, int32_t* steps) {
    if (!h || !phase_ms || !steps) return HUGE_ERR_INVALID_ARG;
    huge_status st = HUGE_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    for (int k = 0; k < kSlots; ++k) {
        if (hipStreamWaitEvent(s, h->ready[k], 0) != hipSuccess ||
            hipStreamWaitEvent(s, h->done[k], 0) != hipSuccess)
            st = HUGE_ERR_HIP;
    }
    if (st == HUGE_OK && hipStreamSynchronize(s) != hipSuccess) st = HUGE_ERR_HIP;
    for (int k = 0; k < HUGE_PHASES; ++k) phase_ms[k] = 0.0;
    auto sum = [&](const std::vector<hipEvent_t>& ev, int per, int used, int first_phase) {
        for (int32_t i = 0; st == HUGE_OK && i < used; ++i) {
            for (int k = 0; k + 1 < per; ++k) {
                float ms = 0.0f;
                if (hipEventElapsedTime(&ms, ev[(size_t)i * per + k],
                                        ev[(size_t)i * per + k + 1]) != hipSuccess) {
                    st = HUGE_ERR_HIP;
                    break;
                }
                phase_ms[first_phase + k] += (double)ms;
            }
        }
    };
    sum(h->prep_ev, kPrepEvents, h->prof_prep, 0);
    sum(h->apply_ev, kApplyEvents, h->prof_apply, 3);
    *steps = h->prof_apply < h->prof_prep ? h->prof_apply : h->prof_prep;
    release_profile(h);
    return st;
}

void huge_destroy(huge_handle* h) { destroy_handle(h); }

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
