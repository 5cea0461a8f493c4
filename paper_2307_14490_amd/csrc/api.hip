// C-ABI host layer of libhuge: argument checks, workspace layout, and the
// launch sequence of each call on the caller's streams.
//
// A batch is prepared, then applied.  Preparing (huge_prepare_step, on the
// caller's preparation stream) validates the batch, draws its negatives and
// groups its rows: k_begin, k_sample (keys, negatives and the digit counts
// of each radix tile, a tile being one sampler workgroup's keys), k_tile_scan
// (the counts' prefixes over tiles), k_radix_pass (occurrences grouped by the
// lowest digits of their key) and k_group (repeated rows and their slots).  These read only the batch, and every one
// of them runs in 256-thread workgroups of few registers, so that they run
// beside the previous batch's apply without evicting its waves.  Applying
// (huge_train_prepared, on the apply stream) runs the fused step and the
// finish kernel (repeated rows, loss).  kSlots grouping slots let two batches
// be prepared ahead; events order the halves: an apply waits for its batch's
// preparation and for the previous apply, a preparation for the apply that
// last used its slot (an apply's completion is recorded only where such a
// wait needs it).
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "../../include/huge.h"
#include "common.hpp"

using namespace huge;

// The workspace of huge_eval_summary_static (32 MiB; its use is described
// where its address is looked up).
constexpr size_t kStaticScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) uint8_t scratch[kStaticScratchBytes];

namespace {

// Events recorded per profiled batch: sampling start and end (after the
// tile prefixes), radix pass start and end, grouping start and end, apply
// start, after the fused kernel, after the finish kernel (repeated rows and
// the loss), and a last one at the same point (the loss has no kernel of
// its own).
constexpr int kProfEvents = 10;
constexpr int kMaxPending = 2;  // prepared batches not yet applied

struct PendingBatch {
    const int32_t* src = nullptr;
    const int32_t* dst = nullptr;
    const int32_t* cc = nullptr;
    const float* w = nullptr;    // float weights in place of cc
    int64_t n = 0;
    uint64_t first_pos = 0;
    hipStream_t gstream = nullptr;  // the stream of its huge_prepare_step
    int prof = -1;               // index of its profile events, or -1
    int bits = kMinDigitBits;    // digit width of its radix pass (buckets 2^bits)
};

}  // namespace

struct huge_handle {
    huge_config cfg;
    void* S;  // rows of cfg.table_dtype
    void* T;
    const uint32_t* thr;
    const int32_t* alias;
    uint8_t* ws;
    size_t ws_bytes;
    Layout lay;
    int key_bits;   // bits of 2N - 1
    int64_t prepared;          // batches prepared
    int64_t applied;           // applies issued
    int last_applied_slot;     // -1 before the first apply
    PendingBatch pending[kSlots];
    hipEvent_t ready[kSlots];    // preparation of the slot's batch complete
    // The completions of applies done_idx and done_idx2 (0-based), recorded
    // on done_stream and done_stream2: an apply's completion implies that of
    // every earlier one, so two events, recorded only where a later wait
    // needs one, serve every such wait, each taking the oldest that suffices.
    // Each record costs the recording kernel a signalled completion (a
    // device-wide cache write-back of several microseconds before the next
    // kernel starts).
    hipEvent_t done_ev = nullptr, done_ev2 = nullptr;
    int64_t done_idx = -1, done_idx2 = -1;
    hipStream_t done_stream = nullptr, done_stream2 = nullptr;
    // phase timing
    std::vector<hipEvent_t> prof_ev;
    std::vector<char> prof_applied;
    int32_t prof_max = 0, prof_next = 0;  // batches to profile; profiled so far
    int32_t prof_every = 1, prof_seen = 0;  // every prof_every-th batch; batches seen
    bool prof_all = false;     // events at every phase boundary, not only the fused kernel
    // the stream of the last apply, so that a wait on it from the same
    // stream is skipped (the stream orders it)
    hipStream_t last_apply_stream = nullptr;
    // calls outside the step that read or write the tables or the shared
    // apply regions (huge_eval_loss, huge_get_rows, huge_probe_rows): the
    // next apply waits for the last of them
    hipEvent_t side_done = nullptr;
    hipStream_t side_stream = nullptr;
    bool side_pending = false;
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
    if (c->table_dtype != HUGE_DTYPE_F32 && c->table_dtype != HUGE_DTYPE_BF16) return false;
    // the atomic scatter adds in float
    if (c->table_dtype == HUGE_DTYPE_BF16 && c->scatter_kind == HUGE_SCATTER_ATOMIC) return false;
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
    const ListCaps caps = list_caps(M);
    L.max_occ = M;
    // radix tiles: the keys of one sampler workgroup each (at most
    // kSampleTiles of them until a tile reaches kSortTile keys)
    const int64_t pmax = sample_tile_positives(K, INT64_MAX / 2);
    L.sort_tiles = (nb + pmax - 1) / pmax;
    if (L.sort_tiles < kSampleTiles) L.sort_tiles = kSampleTiles;
    L.loss_blocks = nb + 1;  // at most one workgroup per positive
    L.cap_short = caps.shorts;
    L.cap_piece = caps.pieces;
    L.cap_comb = caps.combs;
    L.cap_part = caps.parts;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t at = off;
        off = align_up(off + bytes);
        return at;
    };
    for (int s = 0; s < kSlots; ++s) {
        SlotLayout& S = L.slot[s];
        S.ctrl = take(sizeof(Control));
        S.hist = take(sizeof(uint32_t) * kMaxBins);
        if (!sorted) S.neg = take(sizeof(int32_t) * (size_t)(nb * K));
        if (sorted) {
            S.keys0 = take(sizeof(uint32_t) * (size_t)M);
            S.keys1 = take(sizeof(uint32_t) * (size_t)M);
            S.vals1 = take(sizeof(uint32_t) * (size_t)M);
            S.info = take(sizeof(int32_t) * (size_t)M);
            S.tcount = take(sizeof(uint32_t) * (size_t)(L.sort_tiles * kMaxBins));
            S.tprefix = take(sizeof(uint32_t) * (size_t)(L.sort_tiles * kMaxBins));
            S.bstart = take(sizeof(uint32_t) * kMaxBins);
            S.shorts = take(sizeof(uint4) * (size_t)caps.shorts);
            S.pieces = take(sizeof(uint4) * (size_t)caps.pieces);
            S.combs = take(sizeof(uint4) * (size_t)caps.combs);
            S.ccount = take(sizeof(uint32_t) * (size_t)caps.combs);
            S.bcount = take(sizeof(uint4) * kMaxBins);
            S.wstats = take(sizeof(uint32_t) * kMaxBins * 3);
        }
    }
    L.eval_ctrl = take(sizeof(Control));
    L.lossp = take(sizeof(double) * (size_t)L.loss_blocks);
    if (sorted) {
        L.part = take(sizeof(double) * (size_t)caps.parts * (size_t)D);
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
    t.dtype = h->cfg.table_dtype == HUGE_DTYPE_BF16 ? kDtypeBf16 : kDtypeF32;
    return t;
}

#define HIP_TRY(expr)                                   \
    do {                                                \
        if ((expr) != hipSuccess) return HUGE_ERR_HIP;  \
    } while (0)

#define HIP_TRY_ST(expr)                  \
    do {                                  \
        const huge_status st_ = (expr);   \
        if (st_ != HUGE_OK) return st_;   \
    } while (0)

void release_profile(huge_handle* h) {
    for (hipEvent_t e : h->prof_ev)
        if (e) (void)hipEventDestroy(e);
    h->prof_ev.clear();
    h->prof_applied.clear();
    h->prof_max = h->prof_next = h->prof_seen = 0;
    h->prof_every = 1;
}

void destroy_handle(huge_handle* h) {
    if (!h) return;
    release_profile(h);
    for (int s = 0; s < kSlots; ++s)
        if (h->ready[s]) (void)hipEventDestroy(h->ready[s]);
    if (h->done_ev) (void)hipEventDestroy(h->done_ev);
    if (h->done_ev2) (void)hipEventDestroy(h->done_ev2);
    if (h->side_done) (void)hipEventDestroy(h->side_done);
    delete h;
}

huge_status create(const huge_config* cfg, void* S, void* T, const uint32_t* thr,
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
    h->prepared = h->applied = 0;
    h->last_applied_slot = -1;
    for (int s = 0; s < kSlots; ++s) h->ready[s] = nullptr;
    // the events order streams of this device only: a device-scope release
    // suffices (the default one is system-scope)
    const unsigned flags = hipEventDisableTiming | hipEventReleaseToDevice;
    for (int s = 0; s < kSlots + 2; ++s) {
        hipEvent_t* e = s < kSlots ? &h->ready[s] : s == kSlots ? &h->done_ev : &h->done_ev2;
        if (hipEventCreateWithFlags(e, flags) != hipSuccess) {
            *e = nullptr;
            destroy_handle(h);
            return HUGE_ERR_HIP;
        }
    }
    if (hipEventCreateWithFlags(&h->side_done, flags) != hipSuccess) {
        h->side_done = nullptr;
        destroy_handle(h);
        return HUGE_ERR_HIP;
    }
    *out = h;
    return HUGE_OK;
}

// Zero the control blocks and mark every occurrence unrepeated, on the stream.
huge_status reset_workspace(huge_handle* h, hipStream_t s) {
    for (int k = 0; k < kSlots; ++k) {
        HIP_TRY(hipMemsetAsync(h->ws + h->lay.slot[k].ctrl, 0, sizeof(Control), s));
        if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED) {
            HIP_TRY(launch_fill_i32(at<int32_t>(h, h->lay.slot[k].info), -1, h->lay.max_occ, s));
        }
    }
    HIP_TRY(hipMemsetAsync(h->ws + h->lay.eval_ctrl, 0, sizeof(Control), s));
    return HUGE_OK;
}

// `weights`: the batch's co_counts or float weights.
huge_status check_batch_args(huge_handle* h, const int32_t* src, const int32_t* dst,
                             const void* weights, int64_t n) {
    if (!h) return HUGE_ERR_INVALID_ARG;
    if (n < 0 || n > h->cfg.max_batch) return HUGE_ERR_INVALID_ARG;
    if (n > 0 && (!src || !dst || !weights)) return HUGE_ERR_INVALID_ARG;
    return HUGE_OK;
}

// Profile event k of a batch, recorded on s (nothing if it is not profiled).
bool prof_mark(huge_handle* h, const PendingBatch& b, int k, hipStream_t s) {
    if (b.prof < 0) return true;
    if (!h->prof_all && k != 6 && k != 7) return true;  // the fused kernel only
    return hipEventRecord(h->prof_ev[(size_t)b.prof * kProfEvents + k], s) == hipSuccess;
}

// Make s wait for event e recorded on stream `from`, unless that is s itself.
hipError_t wait_on(hipStream_t s, hipEvent_t e, hipStream_t from) {
    if (from == s) return hipSuccess;
    return hipStreamWaitEvent(s, e, 0);
}

// Make s wait until apply i (issued) is complete: nothing on the last apply's
// stream (it follows every apply), the recorded completion if it covers i,
// else a completion recorded now after the last apply.
// Overwrite the older of the two recorded completions with apply idx's.
hipEvent_t take_done(huge_handle* h, int64_t idx, hipStream_t s) {
    if (h->done_idx <= h->done_idx2) {
        h->done_idx = idx;
        h->done_stream = s;
        return h->done_ev;
    }
    h->done_idx2 = idx;
    h->done_stream2 = s;
    return h->done_ev2;
}

hipError_t wait_applied(huge_handle* h, hipStream_t s, int64_t i) {
    if (i < 0 || s == h->last_apply_stream) return hipSuccess;
    // the oldest recorded completion that covers i (a later one would hold s back)
    const bool ok1 = h->done_idx >= i, ok2 = h->done_idx2 >= i;
    if (ok1 && (!ok2 || h->done_idx <= h->done_idx2)) return wait_on(s, h->done_ev, h->done_stream);
    if (ok2) return wait_on(s, h->done_ev2, h->done_stream2);
    hipEvent_t e = take_done(h, h->applied - 1, h->last_apply_stream);
    const hipError_t r = hipEventRecord(e, h->last_apply_stream);
    if (r != hipSuccess) return r;
    return wait_on(s, e, h->last_apply_stream);
}

// A call outside the step on stream s: ordered after the last apply (it
// reads the tables or the shared apply regions) ...
hipError_t side_begin(huge_handle* h, hipStream_t s) {
    if (h->side_pending) {  // and after the previous such call (shared regions)
        const hipError_t e = wait_on(s, h->side_done, h->side_stream);
        if (e != hipSuccess) return e;
    }
    return wait_applied(h, s, h->applied - 1);
}

// ... and the next apply ordered after it.
hipError_t side_end(huge_handle* h, hipStream_t s) {
    const hipError_t e = hipEventRecord(h->side_done, s);
    if (e == hipSuccess) {
        h->side_stream = s;
        h->side_pending = true;
    }
    return e;
}

// The preparation of a batch into the next slot, on stream s: validation,
// negatives and keys, tile counts and prefixes, radix pass, grouping
// (launches only; arguments checked).
huge_status stage_prepare(huge_handle* h, const int32_t* src, const int32_t* dst,
                          const int32_t* cc, const float* w, int64_t n, uint64_t first_pos,
                          hipStream_t s) {
    const int slot = (int)(h->prepared % kSlots);
    const SlotLayout& SL = h->lay.slot[slot];
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, SL.ctrl);
    uint32_t* hist = at<uint32_t>(h, SL.hist);
    const TableArgs t = table_args(h);
    StepArgs a{src, dst, cc, n, first_pos, 0.0f, nullptr};
    a.w = w;
    PendingBatch b;
    b.src = src;
    b.dst = dst;
    b.cc = cc;
    b.w = w;
    b.n = n;
    b.first_pos = first_pos;
    b.gstream = s;
    b.prof = -1;
    if (h->prof_next < h->prof_max) {
        if (h->prof_seen % h->prof_every == 0) b.prof = h->prof_next++;
        h->prof_seen += 1;
    }
    // the slot's previous apply must be complete before its buffers change
    HIP_TRY(wait_applied(h, s, h->prepared - kSlots));
    if (!prof_mark(h, b, 0, s)) return HUGE_ERR_HIP;
    HIP_TRY(launch_begin(ctl, s));
    const bool sorted = h->cfg.scatter_kind == HUGE_SCATTER_SORTED;
    bool ready_recorded = false;
    const int64_t S = 2 + (int64_t)h->cfg.num_neg_per_pos;
    const int64_t m = n * S;
    // the sampler's workgroups write the radix tiles' digit counts
    const int bits = batch_digit_bits(h->key_bits, m);
    const int64_t tile = sample_tile_positives(S - 2, n) * S;
    b.bits = bits;
    HIP_TRY(launch_sample(t, ctl, a, sorted ? nullptr : at<int32_t>(h, SL.neg),
                          sorted ? at<uint32_t>(h, SL.keys0) : nullptr,
                          sorted ? at<uint32_t>(h, SL.tcount) : nullptr, bits, s));
    if (sorted) {
        HIP_TRY(launch_tile_scan(ctl, at<uint32_t>(h, SL.tcount), m, tile, bits,
                                 at<uint32_t>(h, SL.tprefix), hist, s));
        if (!prof_mark(h, b, 1, s) || !prof_mark(h, b, 2, s)) return HUGE_ERR_HIP;
        HIP_TRY(launch_radix_pass(ctl, at<uint32_t>(h, SL.keys0), at<uint32_t>(h, SL.keys1),
                                  at<uint32_t>(h, SL.vals1), m, tile, bits, 0, hist,
                                  at<uint32_t>(h, SL.tprefix), at<uint32_t>(h, SL.bstart), s));
        if (!prof_mark(h, b, 3, s) || !prof_mark(h, b, 4, s)) return HUGE_ERR_HIP;
        const ListCaps caps{L.cap_short, L.cap_piece, L.cap_comb, L.cap_part};
        HIP_TRY(launch_group(ctl, at<uint32_t>(h, SL.keys1), at<uint32_t>(h, SL.vals1), m,
                             h->cfg.num_nodes, hist, at<uint32_t>(h, SL.bstart),
                             at<int32_t>(h, SL.info), at<uint4>(h, SL.shorts),
                             at<uint4>(h, SL.pieces), at<uint4>(h, SL.combs),
                             at<uint32_t>(h, SL.ccount), at<uint4>(h, SL.bcount), caps,
                             at<uint32_t>(h, SL.wstats), 1 << bits, h->key_bits,
                             h->ready[slot], &ready_recorded, s));
        if (!prof_mark(h, b, 5, s)) return HUGE_ERR_HIP;
    } else {
        // the atomic scatter needs no grouping
        for (int k = 1; k <= 5; ++k)
            if (!prof_mark(h, b, k, s)) return HUGE_ERR_HIP;
    }
    // the grouping kernel's completion records `ready` (no packet of its own)
    if (!ready_recorded) HIP_TRY(hipEventRecord(h->ready[slot], s));
    h->pending[slot] = b;
    h->prepared += 1;
    return HUGE_OK;
}

// The apply of the oldest prepared batch on s (launches only).
huge_status apply_next(huge_handle* h, float lr, double* loss_out, hipStream_t s) {
    const int slot = (int)(h->applied % kSlots);
    PendingBatch& b = h->pending[slot];
    const SlotLayout& SL = h->lay.slot[slot];
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, SL.ctrl);
    const TableArgs t = table_args(h);
    StepArgs a{b.src, b.dst, b.cc, b.n, b.first_pos, lr, loss_out};
    a.w = b.w;
    double* lossp = at<double>(h, L.lossp);
    const int64_t m = b.n * (2 + (int64_t)h->cfg.num_neg_per_pos);

    HIP_TRY(wait_on(s, h->ready[slot], b.gstream));
    // applies write the tables and share the apply regions: one at a time
    HIP_TRY(wait_applied(h, s, h->applied - 1));
    // and after the calls outside the step issued since the last apply
    if (h->side_pending) {
        HIP_TRY(wait_on(s, h->side_done, h->side_stream));
        h->side_pending = false;
    }
    int64_t blocks = 0;
    // This apply records its completion only if the newest recorded one is
    // older than apply prepared - (kSlots - 1), one later than what the next
    // preparation needs: with one preparation issued ahead of each apply that
    // is every other apply, and a preparation then waits for the apply it
    // needs or the one after it, never a later one.  The finish kernel's own
    // completion records it.
    const int64_t newest = h->done_idx > h->done_idx2 ? h->done_idx : h->done_idx2;
    const bool record_done = newest < h->prepared - (kSlots - 1);
    hipEvent_t done_e = record_done ? take_done(h, h->applied, s) : nullptr;
    if (h->cfg.scatter_kind == HUGE_SCATTER_SORTED) {
        // the negatives are the sort keys of slots 2 .. K + 1; a profiled
        // step's fused-kernel events (6, 7) are the kernel's own start and
        // completion (no packets of their own)
        const uint32_t stride = 2 + (uint32_t)h->cfg.num_neg_per_pos;
        hipEvent_t ev_start = nullptr, ev_stop = nullptr;
        if (b.prof >= 0) {
            ev_start = h->prof_ev[(size_t)b.prof * kProfEvents + 6];
            ev_stop = h->prof_ev[(size_t)b.prof * kProfEvents + 7];
        }
        HIP_TRY(launch_fused_step(t, ctl, a, at<int32_t>(h, SL.keys0) + 2, stride,
                                  at<int32_t>(h, SL.info), at<float>(h, L.dup), lossp, &blocks,
                                  ev_start, ev_stop, s));
        FinishArgs f;
        // an empty batch is not grouped: no record is read (f.m = 0)
        f.m = m;
        f.shorts = at<uint4>(h, SL.shorts);
        f.pieces = at<uint4>(h, SL.pieces);
        f.combs = at<uint4>(h, SL.combs);
        f.ccount = at<uint32_t>(h, SL.ccount);
        f.dup = at<float>(h, L.dup);
        f.part = at<double>(h, L.part);
        f.caps = ListCaps{L.cap_short, L.cap_piece, L.cap_comb, L.cap_part};
        f.lr = lr;
        f.lossp = lossp;
        f.loss_blocks = blocks;
        f.loss_out = loss_out;
        // the finish kernel's completion records it (no packet of its own)
        HIP_TRY(launch_finish(t, ctl, f, done_e, s));
    } else {
        float* gsrc = at<float>(h, L.gsrc);
        float* coef = at<float>(h, L.coef);
        const int32_t* neg = at<int32_t>(h, SL.neg);
        if (!prof_mark(h, b, 6, s)) return HUGE_ERR_HIP;
        HIP_TRY(launch_atomic_gather(t, ctl, a, neg, gsrc, coef, lossp, &blocks, s));
        if (!prof_mark(h, b, 7, s)) return HUGE_ERR_HIP;
        HIP_TRY(launch_atomic_scatter_T(t, ctl, a, neg, coef, s));
        HIP_TRY(launch_atomic_scatter_S(t, ctl, a, gsrc, s));
        if (loss_out) HIP_TRY(launch_loss_final(ctl, lossp, blocks, loss_out, s));
    }
    if (!prof_mark(h, b, 8, s) || !prof_mark(h, b, 9, s)) return HUGE_ERR_HIP;
    if (record_done && h->cfg.scatter_kind != HUGE_SCATTER_SORTED)
        HIP_TRY(hipEventRecord(done_e, s));
    if (b.prof >= 0) h->prof_applied[(size_t)b.prof] = 1;
    h->last_apply_stream = s;
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

huge_status huge_init_tables(const huge_config* cfg, void* d_S, void* d_T,
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

huge_status huge_attach_tables(const huge_config* cfg, void* d_S, void* d_T,
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

}  // extern "C"

namespace {

huge_status train_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                       const int32_t* d_cc, const float* d_w, int64_t n, uint64_t first_pos_index,
                       float lr, double* d_loss_sum, void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc ? (const void*)d_cc : d_w, n);
    if (st != HUGE_OK) return st;
    if (!isfinite(lr)) return HUGE_ERR_INVALID_ARG;
    if (h->prepared != h->applied) return HUGE_ERR_INVALID_ARG;  // a prepared batch is pending
    hipStream_t s = static_cast<hipStream_t>(stream);
    st = stage_prepare(h, d_src, d_dst, d_cc, d_w, n, first_pos_index, s);
    if (st != HUGE_OK) return st;
    return apply_next(h, lr, d_loss_sum, s);
}

huge_status prepare_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                         const int32_t* d_cc, const float* d_w, int64_t n,
                         uint64_t first_pos_index, void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc ? (const void*)d_cc : d_w, n);
    if (st != HUGE_OK) return st;
    if (h->prepared - h->applied >= kMaxPending) return HUGE_ERR_INVALID_ARG;
    return stage_prepare(h, d_src, d_dst, d_cc, d_w, n, first_pos_index,
                         static_cast<hipStream_t>(stream));
}

huge_status eval_loss(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                      const int32_t* d_cc, const float* d_w, int64_t n, uint64_t first_pos_index,
                      double* d_loss_sum, void* stream) {
    huge_status st = check_batch_args(h, d_src, d_dst, d_cc ? (const void*)d_cc : d_w, n);
    if (st != HUGE_OK) return st;
    if (!d_loss_sum) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Layout& L = h->lay;
    Control* ctl = at<Control>(h, L.eval_ctrl);
    // the loss partials are shared with applies
    HIP_TRY(side_begin(h, s));
    double* lossp = at<double>(h, L.lossp);
    StepArgs a{d_src, d_dst, d_cc, n, first_pos_index, 0.0f, d_loss_sum};
    a.w = d_w;
    HIP_TRY(launch_begin(ctl, s));
    int64_t blocks = 0;
    HIP_TRY(launch_eval(table_args(h), ctl, a, lossp, &blocks, s));
    HIP_TRY(launch_loss_final(ctl, lossp, blocks, d_loss_sum, s));
    HIP_TRY(side_end(h, s));
    return HUGE_OK;
}

}  // namespace

extern "C" {

huge_status huge_train_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                            const int32_t* d_cc, int64_t n, uint64_t first_pos_index, float lr,
                            double* d_loss_sum, void* stream) {
    if (n > 0 && !d_cc) return HUGE_ERR_INVALID_ARG;
    return train_step(h, d_src, d_dst, d_cc, nullptr, n, first_pos_index, lr, d_loss_sum, stream);
}

huge_status huge_train_step_weighted(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                                     const float* d_weight, int64_t n, uint64_t first_pos_index,
                                     float lr, double* d_loss_sum, void* stream) {
    if (n > 0 && !d_weight) return HUGE_ERR_INVALID_ARG;
    return train_step(h, d_src, d_dst, nullptr, d_weight, n, first_pos_index, lr, d_loss_sum,
                      stream);
}

huge_status huge_prepare_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                              const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                              void* stream) {
    if (n > 0 && !d_cc) return HUGE_ERR_INVALID_ARG;
    return prepare_step(h, d_src, d_dst, d_cc, nullptr, n, first_pos_index, stream);
}

huge_status huge_prepare_step_weighted(huge_handle* h, const int32_t* d_src,
                                       const int32_t* d_dst, const float* d_weight, int64_t n,
                                       uint64_t first_pos_index, void* stream) {
    if (n > 0 && !d_weight) return HUGE_ERR_INVALID_ARG;
    return prepare_step(h, d_src, d_dst, nullptr, d_weight, n, first_pos_index, stream);
}

huge_status huge_train_prepared(huge_handle* h, float lr, double* d_loss_sum, void* stream) {
    if (!h || !isfinite(lr)) return HUGE_ERR_INVALID_ARG;
    if (h->applied >= h->prepared) return HUGE_ERR_INVALID_ARG;  // nothing prepared
    return apply_next(h, lr, d_loss_sum, static_cast<hipStream_t>(stream));
}

huge_status huge_eval_loss(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                           const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                           double* d_loss_sum, void* stream) {
    if (n > 0 && !d_cc) return HUGE_ERR_INVALID_ARG;
    return eval_loss(h, d_src, d_dst, d_cc, nullptr, n, first_pos_index, d_loss_sum, stream);
}

huge_status huge_eval_loss_weighted(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                                    const float* d_weight, int64_t n, uint64_t first_pos_index,
                                    double* d_loss_sum, void* stream) {
    if (n > 0 && !d_weight) return HUGE_ERR_INVALID_ARG;
    return eval_loss(h, d_src, d_dst, nullptr, d_weight, n, first_pos_index, d_loss_sum, stream);
}

huge_status huge_cocount_weights(const int32_t* d_hist, int64_t n, int32_t window,
                                 const float* h_dist_weights, float* d_weight, void* stream) {
    if (n < 0 || window < 1 || window > kMaxHistWindow || !h_dist_weights ||
        (n > 0 && (!d_hist || !d_weight)))
        return HUGE_ERR_INVALID_ARG;
    for (int32_t d = 0; d < window; ++d)
        if (!(h_dist_weights[d] >= 0.0f && h_dist_weights[d] <= 3.402823466e38f))
            return HUGE_ERR_INVALID_ARG;
    HIP_TRY(launch_cocount_weights(d_hist, n, window, h_dist_weights, d_weight,
                                   static_cast<hipStream_t>(stream)));
    return HUGE_OK;
}

huge_status huge_get_rows(huge_handle* h, int32_t table, const int64_t* d_ids, int64_t n,
                          float* d_out, void* stream) {
    if (!h || (table != 0 && table != 1) || n < 0) return HUGE_ERR_INVALID_ARG;
    if (n == 0) return HUGE_OK;
    if (!d_ids || !d_out) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(side_begin(h, s));
    HIP_TRY(launch_get_rows(table_args(h), at<Control>(h, h->lay.eval_ctrl), table, d_ids, n,
                            d_out, s));
    HIP_TRY(side_end(h, s));
    return HUGE_OK;
}

huge_status huge_probe_rows(huge_handle* h, const int32_t* d_src, const int32_t* d_dst, int64_t n,
                            uint64_t first_pos_index, void* stream) {
    if (!h || n < 0 || n > h->cfg.max_batch) return HUGE_ERR_INVALID_ARG;
    if (n == 0) return HUGE_OK;
    if (!d_src || !d_dst) return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // the probe rewrites table rows: ordered between applies
    HIP_TRY(side_begin(h, s));
    HIP_TRY(launch_probe(table_args(h), at<Control>(h, h->lay.eval_ctrl), d_src, d_dst, n,
                         first_pos_index, s));
    HIP_TRY(side_end(h, s));
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
                          nullptr, 0, s));
    return HUGE_OK;
}

}  // extern "C"

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

extern "C" {

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
    // every stage issued so far, on any stream
    for (int k = 0; k < kSlots; ++k) HIP_TRY(hipStreamWaitEvent(s, h->ready[k], 0));
    HIP_TRY(wait_applied(h, s, h->applied - 1));
    HIP_TRY(hipStreamWaitEvent(s, h->side_done, 0));
    constexpr int kCtrls = kSlots + 1;
    size_t ctrls[kCtrls];
    for (int k = 0; k < kSlots; ++k) ctrls[k] = h->lay.slot[k].ctrl;
    ctrls[kSlots] = h->lay.eval_ctrl;
    Control got[kCtrls];
    for (int k = 0; k < kCtrls; ++k) {
        Control* c = at<Control>(h, ctrls[k]);
        HIP_TRY(hipMemcpyAsync(&got[k], c, sizeof(Control), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemsetAsync(&c->error, 0, sizeof(uint32_t), s));
        HIP_TRY(hipMemsetAsync(&c->site, 0, sizeof(uint32_t), s));
    }
    HIP_TRY(hipStreamSynchronize(s));
    uint32_t first = 0, site = 0;
    for (int k = 0; k < kCtrls; ++k) {
        if (!first) first = got[k].error;
        if (!site) site = got[k].site;
    }
    if (site != 0 && getenv("HUGE_DEBUG") != nullptr)
        fprintf(stderr, "libhuge: internal check %u failed\n", site);
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
        HIP_TRY(wait_applied(h, s, h->applied - 1));
        const int64_t m = h->pending[slot].n * (2 + (int64_t)h->cfg.num_neg_per_pos);
        // k_group writes the counts of every bucket when the batch is not empty
        const int64_t buckets = m > 0 ? ((int64_t)1 << h->pending[slot].bits) : 0;
        std::vector<uint32_t> w((size_t)buckets * 3);
        if (buckets > 0)
            HIP_TRY(hipMemcpyAsync(w.data(), h->ws + h->lay.slot[slot].wstats,
                                   w.size() * sizeof(uint32_t), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        a = b = c = 0;
        for (int64_t i = 0; i < buckets; ++i) {
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

huge_status huge_profile_begin(huge_handle* h, int32_t max_steps, int32_t all_phases,
                               int32_t every) {
    if (!h || max_steps < 1 || max_steps > 1000000) return HUGE_ERR_INVALID_ARG;
    if (all_phases != 0 && all_phases != 1) return HUGE_ERR_INVALID_ARG;
    if (every < 1 || every > 1000000) return HUGE_ERR_INVALID_ARG;
    release_profile(h);
    h->prof_all = all_phases != 0;
    h->prof_every = every;
    h->prof_ev.assign((size_t)max_steps * kProfEvents, nullptr);
    h->prof_applied.assign((size_t)max_steps, 0);
    for (hipEvent_t& e : h->prof_ev) {
        if (hipEventCreateWithFlags(&e, hipEventReleaseToDevice) != hipSuccess) {
            e = nullptr;
            release_profile(h);
            return HUGE_ERR_HIP;
        }
    }
    h->prof_max = max_steps;
    return HUGE_OK;
}

huge_status huge_profile_end(huge_handle* h, void* stream, double* phase_ms, int32_t* steps) {
    if (!h || !phase_ms || !steps) return HUGE_ERR_INVALID_ARG;
    huge_status st = HUGE_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    for (int k = 0; k < kSlots && st == HUGE_OK; ++k)
        if (hipStreamWaitEvent(s, h->ready[k], 0) != hipSuccess) st = HUGE_ERR_HIP;
    if (st == HUGE_OK && wait_applied(h, s, h->applied - 1) != hipSuccess) st = HUGE_ERR_HIP;
    if (st == HUGE_OK && hipStreamSynchronize(s) != hipSuccess) st = HUGE_ERR_HIP;
    for (int k = 0; k < HUGE_PHASES; ++k) phase_ms[k] = 0.0;
    // phase p lasts from event first[p] to event last[p] of a batch
    static const int first[HUGE_PHASES] = {0, 2, 4, 6, 7, 8};
    static const int last[HUGE_PHASES] = {1, 3, 5, 7, 8, 9};
    int32_t counted = 0;
    for (int32_t i = 0; st == HUGE_OK && i < h->prof_next; ++i) {
        if (!h->prof_applied[(size_t)i]) continue;
        const bool sorted = h->cfg.scatter_kind == HUGE_SCATTER_SORTED;
        for (int p = 0; p < HUGE_PHASES; ++p) {
            if (!sorted && (p == 1 || p == 2)) continue;  // no radix pass or grouping
            if (!h->prof_all && p != 3) continue;         // only the fused kernel
            float ms = 0.0f;
            if (hipEventElapsedTime(&ms, h->prof_ev[(size_t)i * kProfEvents + first[p]],
                                    h->prof_ev[(size_t)i * kProfEvents + last[p]]) !=
                hipSuccess) {
                st = HUGE_ERR_HIP;
                break;
            }
            phase_ms[p] += (double)ms;
        }
        ++counted;
    }
    *steps = counted;
    release_profile(h);
    return st;
}

// ---------------------------------------------------------------------------
// Embedding evaluation.  The summary and the nearest-row search each lay out
// their regions from the start of the caller's workspace (calls on a stream
// run one after the other).
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

struct SummaryLayout {
    size_t ctrl, keys_a, keys_b, tcount, tprefix, hist, part, total;
};

SummaryLayout summary_layout(int64_t max_pairs) {
    SummaryLayout L;
    const size_t n = (size_t)(max_pairs > 0 ? max_pairs : 1);
    const size_t tiles = (n + kSortTile - 1) / kSortTile;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align_up(off + bytes);
        return at;
    };
    L.ctrl = take(sizeof(Control));
    L.keys_a = take(sizeof(uint32_t) * n);
    L.keys_b = take(sizeof(uint32_t) * n);
    L.tcount = take(sizeof(uint32_t) * tiles * kMaxBins);
    L.tprefix = take(sizeof(uint32_t) * tiles * kMaxBins);
    L.hist = take(sizeof(uint32_t) * kMaxBins);
    L.part = take(sizeof(double) * kEvalSumBlocks * 4);
    L.total = off;
    return L;
}

struct KnnLayout {
    size_t qn, qn2, qid, partial, tau, cnt, gate, cand, total;
};

KnnLayout knn_layout(int64_t num_rows, int32_t dim, int32_t k) {
    KnnLayout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align_up(off + bytes);
        return at;
    };
    L.qn = take(sizeof(float) * kKnnPass * (size_t)dim);
    L.qn2 = take(sizeof(float) * kKnnPass);
    L.qid = take(sizeof(int32_t) * kKnnPass);
    // the most lists: one query block, every wave its own list
    L.partial =
        take(sizeof(uint64_t) * (size_t)knn_lists(num_rows, dim, 1) * kKnnPass * (size_t)k);
    // the threshold scans' bounds, counts, gate and candidate lists
    L.tau = take(sizeof(float) * kKnnPass);
    L.cnt = take(sizeof(uint32_t) * kKnnPass);
    L.gate = take(sizeof(int32_t));
    L.cand = take(sizeof(uint64_t) * kKnnPass * (size_t)kKnnCandCap);
    L.total = off;
    return L;
}

bool eval_table_ok(int64_t num_rows, int32_t dim) {
    return num_rows >= 1 && num_rows <= 0x7FFFFFFF && dim >= 4 && dim <= kMaxDim && dim % 4 == 0;
}

bool eval_graph_ok(int64_t num_nodes, int64_t num_edges) {
    return num_nodes >= 1 && num_nodes <= 0x7FFFFFFF && num_edges >= 0;
}

// The workspace of huge_eval_summary_static: a fixed array in device memory,
// one per device (the runtime creates it on each device when the code object
// is loaded there; it stays until the process ends), for callers that cannot
// allocate.  Host code never passes the array's name to a kernel (on the host
// it is a stand-in, not a device address): the address comes from
// hipGetSymbolAddress, looked up once per device with that device current.
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

hipError_t static_scratch(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

// The argument checks of the summary (all but the workspace).
huge_status eval_summary_args(const float* d_dist, int64_t n_edge, int64_t n_non,
                              const double* h_quantiles, int32_t n_quantiles,
                              const double* d_out) {
    if (n_edge < 0 || n_non < 0 || n_edge + n_non > 0x7FFFFFFF || !d_out || n_quantiles < 0 ||
        n_quantiles > kEvalMaxQuantiles || (n_quantiles > 0 && !h_quantiles) ||
        (n_edge + n_non > 0 && !d_dist))
        return HUGE_ERR_INVALID_ARG;
    for (int32_t i = 0; i < n_quantiles; ++i)
        if (!(h_quantiles[i] >= 0.0 && h_quantiles[i] <= 100.0)) return HUGE_ERR_INVALID_ARG;
    return HUGE_OK;
}

// The summary on a workspace of ws_bytes at d_workspace (launches only).
huge_status eval_summary(const float* d_dist, int64_t n_edge, int64_t n_non,
                         const double* h_quantiles, int32_t n_quantiles, double* d_out,
                         void* d_workspace, size_t ws_bytes, void* stream) {
    const huge_status st = eval_summary_args(d_dist, n_edge, n_non, h_quantiles, n_quantiles,
                                             d_out);
    if (st != HUGE_OK) return st;
    if (!d_workspace) return HUGE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(d_workspace) % kAlign != 0) return HUGE_ERR_WORKSPACE;
    const SummaryLayout L = summary_layout(n_edge + n_non);
    if (ws_bytes < L.total) return HUGE_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t* ws = static_cast<uint8_t*>(d_workspace);
    Control* ctl = reinterpret_cast<Control*>(ws + L.ctrl);
    uint32_t* ka = reinterpret_cast<uint32_t*>(ws + L.keys_a);
    uint32_t* kb = reinterpret_cast<uint32_t*>(ws + L.keys_b);
    uint32_t* tcount = reinterpret_cast<uint32_t*>(ws + L.tcount);
    uint32_t* tprefix = reinterpret_cast<uint32_t*>(ws + L.tprefix);
    uint32_t* hist = reinterpret_cast<uint32_t*>(ws + L.hist);
    double* part = reinterpret_cast<double*>(ws + L.part);
    HIP_TRY(launch_begin(ctl, s));
    HIP_TRY(launch_eval_sums(d_dist, n_edge, n_edge + n_non, part, d_out, s));
    // each set sorted by its float bit patterns: four stable passes of 8 bits
    const int64_t first[2] = {0, n_edge};
    const int64_t count[2] = {n_edge, n_non};
    for (int set = 0; set < 2; ++set) {
        const int64_t m = count[set];
        HIP_TRY(launch_eval_keys(d_dist + first[set], m, ka, s));
        for (int pass = 0; pass < 4; ++pass) {
            uint32_t* src = pass % 2 == 0 ? ka : kb;
            uint32_t* dst = pass % 2 == 0 ? kb : ka;
            HIP_TRY(launch_tile_count(ctl, src, m, 8, 8 * pass, tcount, s));
            HIP_TRY(launch_tile_scan(ctl, tcount, m, kSortTile, 8, tprefix, hist, s));
            HIP_TRY(launch_radix_pass(ctl, src, dst, nullptr, m, kSortTile, 8, 8 * pass, hist,
                                      tprefix, nullptr, s));
        }
        HIP_TRY(launch_eval_quantiles(ka, d_out + set, h_quantiles, n_quantiles,
                                      d_out + 5 + set * n_quantiles, s));
    }
    return HUGE_OK;
}

huge_status eval_knn(const float* d_table, int64_t num_rows, int32_t dim,
                     const int32_t* d_queries, int32_t n_queries, int32_t k, int32_t* d_ids,
                     float* d_dist, void* d_workspace, size_t ws_bytes, bool lists_only,
                     int32_t* d_status, void* stream) {
    if (!d_table || !d_status || !eval_table_ok(num_rows, dim) || n_queries < 0 || k < 1 ||
        k > kKnnMaxK || knn_pass_queries(dim) < 32 || !d_workspace ||
        (n_queries > 0 && (!d_queries || !d_ids || !d_dist)))
        return HUGE_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(d_workspace) % kAlign != 0) return HUGE_ERR_WORKSPACE;
    const KnnLayout L = knn_layout(num_rows, dim, k);
    if (ws_bytes < L.total) return HUGE_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(launch_eval_status_clear(d_status, s));
    if (n_queries == 0) return HUGE_OK;
    uint8_t* ws = static_cast<uint8_t*>(d_workspace);
    KnnBuffers B;
    B.qn = reinterpret_cast<float*>(ws + L.qn);
    B.qn2 = reinterpret_cast<float*>(ws + L.qn2);
    B.qid = reinterpret_cast<int32_t*>(ws + L.qid);
    B.partial = reinterpret_cast<uint64_t*>(ws + L.partial);
    B.tau = reinterpret_cast<float*>(ws + L.tau);
    B.cnt = reinterpret_cast<uint32_t*>(ws + L.cnt);
    B.gate = reinterpret_cast<int32_t*>(ws + L.gate);
    B.cand = reinterpret_cast<uint64_t*>(ws + L.cand);
    HIP_TRY(launch_knn(d_table, num_rows, dim, d_queries, n_queries, k, d_ids, d_dist, B,
                       lists_only, d_status, s));
    return HUGE_OK;
}

}  // namespace

extern "C" {

size_t huge_eval_workspace_bytes(int64_t max_pairs, int64_t num_rows, int32_t dim, int32_t k) {
    if (max_pairs < 0 || max_pairs > 0x7FFFFFFF || !eval_table_ok(num_rows, dim) || k < 1 ||
        k > kKnnMaxK)
        return 0;
    const size_t a = summary_layout(max_pairs).total;
    const size_t b = knn_layout(num_rows, dim, k).total;
    return a > b ? a : b;
}

huge_status huge_eval_pairs(const int64_t* d_offsets, const int32_t* d_neighbors,
                            int64_t num_nodes, int64_t num_edges, uint64_t seed, int64_t n_edge,
                            int64_t n_non, int32_t max_tries, int32_t* d_u, int32_t* d_v,
                            int32_t* d_status, void* stream) {
    if (!d_offsets || !d_status || !eval_graph_ok(num_nodes, num_edges) || n_edge < 0 ||
        n_non < 0 || max_tries < 1 || (n_edge > 0 && num_edges == 0) ||
        (num_edges > 0 && !d_neighbors) || n_edge + n_non > 0x7FFFFFFF ||
        (n_edge + n_non > 0 && (!d_u || !d_v)))
        return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(launch_eval_status_clear(d_status, s));
    HIP_TRY(launch_eval_pairs(d_offsets, d_neighbors, num_nodes, num_edges, seed, n_edge, n_non,
                              max_tries, d_u, d_v, d_status, s));
    return HUGE_OK;
}

huge_status huge_eval_distances(const float* d_table, int64_t num_rows, int32_t dim,
                                const int32_t* d_u, const int32_t* d_v, int64_t n,
                                float* d_dist, int32_t* d_status, void* stream) {
    if (!d_table || !d_status || !eval_table_ok(num_rows, dim) || n < 0 ||
        (n > 0 && (!d_u || !d_v || !d_dist)))
        return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(launch_eval_status_clear(d_status, s));
    HIP_TRY(launch_eval_dist(d_table, num_rows, dim, d_u, d_v, n, d_dist, d_status, s));
    return HUGE_OK;
}

huge_status huge_eval_summary(const float* d_dist, int64_t n_edge, int64_t n_non,
                              const double* h_quantiles, int32_t n_quantiles, double* d_out,
                              void* d_workspace, size_t ws_bytes, void* stream) {
    return eval_summary(d_dist, n_edge, n_non, h_quantiles, n_quantiles, d_out, d_workspace,
                        ws_bytes, stream);
}

huge_status huge_eval_summary_static(const float* d_dist, int64_t n_edge, int64_t n_non,
                                     const double* h_quantiles, int32_t n_quantiles,
                                     double* d_out, void* stream) {
    const huge_status st = eval_summary_args(d_dist, n_edge, n_non, h_quantiles, n_quantiles,
                                             d_out);
    if (st != HUGE_OK) return st;
    if (summary_layout(n_edge + n_non).total > kStaticScratchBytes) return HUGE_ERR_WORKSPACE;
    void* ws = nullptr;
    if (static_scratch(&ws) != hipSuccess) return HUGE_ERR_HIP;
    return eval_summary(d_dist, n_edge, n_non, h_quantiles, n_quantiles, d_out, ws,
                        kStaticScratchBytes, stream);
}

huge_status huge_eval_knn(const float* d_table, int64_t num_rows, int32_t dim,
                          const int32_t* d_queries, int32_t n_queries, int32_t k,
                          int32_t* d_ids, float* d_dist, void* d_workspace, size_t ws_bytes,
                          int32_t* d_status, void* stream) {
    return eval_knn(d_table, num_rows, dim, d_queries, n_queries, k, d_ids, d_dist, d_workspace,
                    ws_bytes, false, d_status, stream);
}

huge_status huge_eval_knn_lists(const float* d_table, int64_t num_rows, int32_t dim,
                                const int32_t* d_queries, int32_t n_queries, int32_t k,
                                int32_t* d_ids, float* d_dist, void* d_workspace,
                                size_t ws_bytes, int32_t* d_status, void* stream) {
    return eval_knn(d_table, num_rows, dim, d_queries, n_queries, k, d_ids, d_dist, d_workspace,
                    ws_bytes, true, d_status, stream);
}

huge_status huge_eval_recall(const int64_t* d_offsets, const int32_t* d_neighbors,
                             int64_t num_nodes, int64_t num_edges, const int32_t* d_queries,
                             int32_t n_queries, const int32_t* d_ids, int32_t k,
                             double* d_recall, int32_t* d_status, void* stream) {
    if (!d_offsets || !d_status || !eval_graph_ok(num_nodes, num_edges) || n_queries < 0 ||
        k < 1 || k > 64 || (num_edges > 0 && !d_neighbors) ||
        (n_queries > 0 && (!d_queries || !d_ids || !d_recall)))
        return HUGE_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIP_TRY(launch_eval_status_clear(d_status, s));
    HIP_TRY(launch_eval_recall(d_offsets, d_neighbors, num_nodes, num_edges, d_queries, n_queries,
                               d_ids, k, d_recall, d_status, s));
    return HUGE_OK;
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
