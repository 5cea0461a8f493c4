// Internal declarations shared by the kernels and the host layer of libhuge.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace huge {

// ---------------------------------------------------------------------------
// Compile-time constants
// ---------------------------------------------------------------------------
constexpr int kBlock = 256;            // threads per workgroup (4 wave64)
constexpr int kMinDigitBits = 8;       // digit widths of the LSD radix sort: 8 to 10 bits,
constexpr int kMaxDigitBits = 10;      // the same in every pass of a sort
constexpr int kMaxBins = 1 << kMaxDigitBits;
constexpr int kMaxPasses = 4;          // keys < 2^32
constexpr int kSortTile = 8192;        // keys per radix-pass tile
// Every kernel of the grouping (tile counts, their prefixes, the radix pass,
// the per-bucket grouping) runs in workgroups of kBlock threads within the
// HUGE_BESIDE register budget, so that it runs beside the fused step without
// evicting any of the step's waves.
constexpr int kScanDigits = 4;         // digits per tile-prefix workgroup
// Register budget of the kernels that run beside the fused step: at most 64
// VGPRs (the budget of eight waves per SIMD).  With the fused step at five
// waves of 88 VGPRs per SIMD (440 of 512), one such wave per SIMD fits beside
// them.
#define HUGE_BESIDE __attribute__((amdgpu_waves_per_eu(8, 8)))
// The same at 72 VGPRs (seven waves per SIMD), the most that fits beside the
// fused step's five waves, for the per-bucket grouping, which needs them.
#define HUGE_BESIDE_72 __attribute__((amdgpu_waves_per_eu(7, 7)))
// Per-bucket grouping (k_group): chunks of kGroupChunk keys (kGroupItems
// consecutive keys per thread); an LDS hash table of kGroupSlots slots counts
// the repeated keys of a key range; a range with more than 3/4 of the slots
// in distinct keys is split by further hash bits.  Where a bucket's keys
// differ in at most kBitmapBits bits, an LDS bitmap of them first marks the
// keys that occur more than once, and only those enter the table.  The first
// pass copies up to kGroupCacheKeys keys and kGroupCacheVals occurrence
// indices of a bucket to LDS; later passes read them there.
constexpr int kGroupItems = 4;
constexpr int kGroupChunk = kBlock * kGroupItems;     // 1024 keys per chunk
constexpr int kGroupTableBits = 12;
constexpr int kGroupSlots = 1 << kGroupTableBits;     // 4096 slots, 32 KB
constexpr int kGroupCacheKeys = 8192;                 // 32 KB
constexpr int kGroupCacheVals = 4096;                 // 16 KB
constexpr int kBitmapBits = 18;        // two 32 KB bitmaps (seen, repeated)
// Embedding evaluation
constexpr int kEvalMaxQuantiles = 128;  // percentiles per summary
constexpr int kKnnWaves = 4;            // waves of a nearest-row workgroup (dim > 128)
constexpr int kKnnWavesR = 8;           // the same with the queries in registers (dim <= 128)
constexpr int kKnnMaxK = 32;            // nearest rows per query, at most
constexpr int kKnnDimChunk = 128;       // dimensions per MFMA pass over a row tile
constexpr int kKnnQueryFloats = 16896;  // LDS floats for the queries of a pass (66 KB)
constexpr int kKnnPass = 128;           // queries per pass over the table, at most
constexpr int kKnnGrid = 256;           // nearest-row workgroups (one per CU)
constexpr int kKnnMergeCap = 8192;      // keys sorted together by the merge
// Threshold scans of the nearest-row search (dim <= 128)
constexpr int kKnnScanWaves = 4;        // waves of a scan workgroup (two workgroups per CU)
constexpr int kKnnScanGrid = 512;       // scan workgroups, at most
constexpr int kKnnCandCap = 8192;       // candidate keys kept per query and scan
constexpr int kKnnStageTiles = 256;     // row tiles of the first (coarsest) scan, at most
constexpr int kKnnStageGrowth = 32;     // tile stride of a scan over that of the next
constexpr int kKnnSelectThreads = 1024; // threads of a candidate selection workgroup
constexpr uint32_t kShortRun = 32;     // repeated rows with at most this many occurrences are
                                       // summed by one thread group
constexpr uint32_t kPiece = 256;       // occurrences summed by one workgroup task
constexpr int kSamplePos = 512;        // positives per sampler workgroup
constexpr int kNegBlock = 8;           // negatives whose rows are in flight together
constexpr int kMaxNeg = 64;
constexpr int kMaxDim = 1024;
// Random-walk sampler: one workgroup holds a seed's walks and pairs in LDS.
constexpr int kWalkMaxWalks = 1024;    // walks per seed
constexpr int kWalkMaxNodes = 8192;    // walks x (steps + 1)
constexpr int kWalkMaxPairs = 4096;    // co-occurrence pairs of one seed
constexpr int kWalkMaxSteps = 64;
constexpr int kWalkMaxWindow = 32;

// Status bits of a step (Control::step_bad) and the sticky error code.
constexpr uint32_t kBadId = 1u;
constexpr uint32_t kBadCount = 2u;
constexpr uint32_t kBadInternal = 4u;  // a bounded wait expired or an index check failed

// Device-side control block, at the start of the workspace.
struct Control {
    uint32_t step_bad;               // this call's input is invalid: skip all writes
    uint32_t error;                  // first error since huge_check (kBadId/kBadCount)
    uint32_t site;                   // first failed internal check (a kSite* code)
    uint32_t nshort;                 // short-run records of the batch (its grouping's)
    uint32_t npiece;                 // its pieces
    uint32_t pad[11];
};

// Internal checks (kBadInternal), recorded in Control::site.
enum InternalSite : uint32_t {
    kSiteRadixDest = 3,
    kSiteGroupBucket = 4,
    kSiteGroupDepth = 5,
    kSiteGroupLists = 6,
    kSiteGroupLookup = 7,
    kSiteGroupPlace = 8,
    kSiteStepIds = 9,
    kSiteAtomicIds = 10,
    kSiteGroupBits = 11,
    kSiteFinishComb = 12,
};

// Byte offsets of the workspace regions (all 256-byte aligned).
//
// A batch is processed in two halves: grouping (validation, negatives, sort,
// run marking) and applying (gather, loss, updates).  Grouping never touches
// the tables, so the grouping of later batches may run on another stream
// while the current one is applied: each grouping slot has its own regions;
// the apply regions are shared (applies are ordered).
struct SlotLayout {
    size_t ctrl = 0;     // Control
    size_t hist = 0;     // u32 [kMaxBins] occurrences per bucket (digit)
    size_t neg = 0;      // i32 [max_batch * K] (atomic scatter; the sorted one reads keys0)
    // sorted scatter
    size_t keys0 = 0;    // u32 [M] keys in occurrence order
    size_t keys1 = 0;    // u32 [M] keys grouped by their lowest digit
    size_t vals1 = 0;    // u32 [M] their occurrence indices
    size_t info = 0;     // i32 [M]: -1, or the duplicate-buffer slot of an occurrence of a
                         // repeated row (-1 between batches: the fused step resets it)
    size_t tcount = 0;   // u32 [sort_tiles * kMaxBins] occurrences per tile and digit
    size_t tprefix = 0;  // u32 [sort_tiles * kMaxBins] the same summed over earlier tiles
    size_t bstart = 0;   // u32 [kMaxBins] first position of each bucket
    // repeated-row records: short runs and pieces in one list each (a range
    // of the grouping appends at positions reserved from Control::nshort,
    // ::npiece); bucket b (first position s0, n items) writes its combine
    // records at [s0 / 256, ...) and partial slots from s0 / 128 (ListCaps
    // says why they fit) and its counts to bcount[b]
    size_t shorts = 0;   // uint4 [cap_short] {start, len, key, 0}
    size_t pieces = 0;   // uint4 [cap_piece] {start, len, key, 0 or combine record index + 1}
    size_t combs = 0;    // uint4 [cap_comb] {key, first partial, partials, first slot}
    size_t ccount = 0;   // u32 [cap_comb] pieces of the row summed so far
    size_t bcount = 0;   // uint4 [kMaxBins] {short runs, pieces, combines, 0} per bucket
    size_t wstats = 0;   // u32 [kMaxBins * 3] distinct S, distinct T, repeated occurrences
};

constexpr int kSlots = 4;  // grouping slots: the applied batch, the next, one being prepared
                           // and one more, so that a preparation can wait for an apply one
                           // earlier than the last while completions are recorded every
                           // other step (the wait paces the preparation: with six slots and
                           // one completion in five it ran onto the finish kernel and the
                           // step slowed from 0.457 to 0.463 ms)

struct Layout {
    SlotLayout slot[kSlots];
    size_t eval_ctrl = 0;  // Control of huge_eval_loss
    size_t lossp = 0;      // double [loss_blocks]
    // sorted scatter
    size_t part = 0;     // f64 [cap_part * D] partial sums of the pieces of long runs
    size_t dup = 0;      // f32 [M * D] per-occurrence contributions of repeated rows
    // atomic scatter
    size_t gsrc = 0;     // f32 [max_batch * D] source-row gradients
    size_t coef = 0;     // f32 [max_batch * (1 + K)]
    size_t total = 0;
    int64_t max_occ = 0;       // M = max_batch * (2 + K)
    int64_t sort_tiles = 0;
    int64_t loss_blocks = 0;
    uint32_t cap_short = 0, cap_piece = 0, cap_comb = 0, cap_part = 0;
};

// Record regions for M occurrences.  Bucket b holds n_b items from position
// s0_b; it writes at most floor(n_b / 2) short runs (a repeated row has >= 2
// occurrences), floor(n_b / 16) pieces (a piece is a whole run of
// kShortRun+1 .. kPiece occurrences, or one of the ceil(c / kPiece) <= c / 16
// pieces of a run of c > kPiece), floor(n_b / 256) combine records (a
// combined row has more than kPiece occurrences) and floor(n_b / 128) partial
// sums (ceil(c / kPiece) <= c / 128 of them per combined row); since
// floor(x + y) >= floor(x) + floor(y), the region of bucket b starting at
// floor(s0_b / q) ends before that of bucket b + 1.
constexpr uint32_t kShortDiv = 2, kPieceDiv = 16, kCombDiv = 256, kPartDiv = 128;
struct ListCaps {
    uint32_t shorts, pieces, combs, parts;
};

inline ListCaps list_caps(int64_t M) {
    return {(uint32_t)(M / kShortDiv + 1), (uint32_t)(M / kPieceDiv + 1),
            (uint32_t)(M / kCombDiv + 1), (uint32_t)(M / kPartDiv + 1)};
}

// Bucketing of keys below 2^key_bits: one radix pass on the lowest digit;
// the grouping of each bucket resolves the remaining key_bits - bits bits.
// Digit width of a batch of m keys below 2^key_bits: the narrowest width in
// kMinDigitBits..kMaxDigitBits whose buckets hold about kBucketTarget keys on
// average (a grouping workgroup's fixed work per bucket is then spread over
// as many keys as in a large batch), but no narrower than leaves the bits
// above the digit within the grouping's bitmap (kBitmapBits) where the key
// width allows.
constexpr int64_t kBucketTarget = 2048;
inline int batch_digit_bits(int key_bits, int64_t m) {
    int bits = kMinDigitBits;
    while (bits < kMaxDigitBits && (m >> bits) > kBucketTarget) ++bits;
    int floor_bits = key_bits - kBitmapBits;
    if (floor_bits > kMaxDigitBits) floor_bits = kMaxDigitBits;
    return bits > floor_bits ? bits : floor_bits;
}

// Element type of the tables (the public HUGE_DTYPE_* values).
enum : int32_t { kDtypeF32 = 0, kDtypeBf16 = 1 };

// A bfloat16 element: the upper 16 bits of an IEEE binary32.
typedef uint16_t bf16_t;

// Rows handled per workgroup: G lanes per row, C float4 per lane.
struct RowShape {
    int G;
    int C;
};

inline RowShape row_shape(int dim) {
    int q = dim / 4;
    int G = 1;
    while (G < q && G < 64) G <<= 1;
    int C = (q + G - 1) / G;
    return {G, C};
}

// Rows of bf16 tables whose width is a multiple of 8, in 8-element units:
// G lanes per row (a power of two <= 64), U units per lane.
struct PairShape {
    int G;
    int U;
};

inline PairShape pair_shape(int dim) {
    const int nu = dim / 8;
    int G = 1;
    while (G < nu && G < 64) G <<= 1;
    return {G, (nu + G - 1) / G};
}

// The fused step and the probe take the unit layout for these tables.
inline bool uses_pairs(int32_t dtype, int dim) { return dtype == kDtypeBf16 && dim % 8 == 0; }

struct StepArgs {
    const int32_t* src;
    const int32_t* dst;
    const int32_t* cc;         // integer co_counts, or
    int64_t n;
    uint64_t first_pos;
    float lr;
    double* loss_out;
    const float* w = nullptr;  // a float weight per positive (then cc is unused)
};

struct TableArgs {
    void* S;               // float or bf16_t rows, as dtype says
    void* T;
    int64_t N;
    int32_t D;
    int32_t K;
    uint64_t seed;
    const uint32_t* thr;   // alias thresholds or nullptr (uniform)
    const int32_t* alias;
    int32_t dtype;         // kDtypeF32 or kDtypeBf16
};

struct WalkArgs {
    const int64_t* off;  // CSR offsets, num_nodes + 1
    const int32_t* nbr;  // CSR neighbours, num_edges
    int64_t num_nodes;
    int64_t num_edges;
    int32_t walks;       // walks per seed (gamma)
    int32_t steps;       // steps per walk (k)
    int32_t window;      // largest co-occurrence distance
    int32_t seed_only;   // pairs (seed, w_t) only
    uint64_t seed;       // Philox key
    int64_t first_seed;
    int64_t num_seeds;
};

// ---------------------------------------------------------------------------
// Launchers (each defined next to its kernels).  All return hipError_t of the
// launch.
// ---------------------------------------------------------------------------
hipError_t launch_init(const TableArgs& t, float half_width, hipStream_t s);
hipError_t launch_get_rows(const TableArgs& t, Control* ctl, int32_t table, const int64_t* ids,
                           int64_t n, float* out, hipStream_t s);
hipError_t launch_begin(Control* ctl, hipStream_t s);
// Positives per sampler workgroup when it writes sort keys for a batch of n
// positives: its keys, (2 + K) per positive, are one radix tile.  A batch
// gets about kSampleTiles workgroups (one per CU) until a tile reaches
// kSortTile keys.
constexpr int64_t kSampleTiles = 256;
inline int64_t sample_tile_positives(int64_t K, int64_t n) {
    const int64_t pmax = kSortTile / (2 + K);
    int64_t p = (n + kSampleTiles - 1) / kSampleTiles;
    if (p < 1) p = 1;
    return p < pmax ? p : pmax;
}
// Validation, negatives into neg (if not null) and, with keys, the sort key
// of every occurrence and the counts of their lowest `bits` bits per
// workgroup into tcount[workgroup * 2^bits + digit]: a workgroup takes
// sample_tile_positives(K, n) positives then, else kSamplePos.
hipError_t launch_sample(const TableArgs& t, Control* ctl, const StepArgs& a, int32_t* neg,
                         uint32_t* keys, uint32_t* tcount, int bits, hipStream_t s);
// Bucketing of m keys by `bits` bits at `shift` in tiles of `tile` keys
// (at most kSortTile): per-tile digit counts, their sums over earlier tiles
// and the bucket sizes (hist), then the stable scatter into bucket order (one
// pass of an LSD radix sort); bstart (if not null) receives the first
// position of each bucket.
hipError_t launch_tile_count(Control* ctl, const uint32_t* keys, int64_t m, int bits, int shift,
                             uint32_t* tcount, hipStream_t s);
hipError_t launch_tile_scan(Control* ctl, const uint32_t* tcount, int64_t m, int64_t tile,
                            int bits, uint32_t* tprefix, uint32_t* hist, hipStream_t s);
hipError_t launch_radix_pass(Control* ctl, const uint32_t* keys_in, uint32_t* keys_out,
                             uint32_t* vals_out, int64_t m, int64_t tile, int bits, int shift,
                             const uint32_t* hist, const uint32_t* tprefix, uint32_t* bstart,
                             hipStream_t s);
// stop (if not null) is recorded by the kernel's completion; *launched says
// whether a kernel was launched (an empty batch launches none).
hipError_t launch_group(Control* ctl, const uint32_t* keys, const uint32_t* vals, int64_t m,
                        int64_t N, const uint32_t* hist, const uint32_t* bstart, int32_t* info,
                        uint4* shorts, uint4* pieces, uint4* combs, uint32_t* ccount,
                        uint4* bcount, ListCaps caps, uint32_t* wstats, int bins, int key_bits,
                        hipEvent_t stop, bool* launched, hipStream_t s);
// Negative k of positive i: neg[i * neg_stride + k].
// start, stop (if not null): recorded at the kernel's start and completion.
hipError_t launch_fused_step(const TableArgs& t, Control* ctl, const StepArgs& a,
                             const int32_t* neg, uint32_t neg_stride, int32_t* info, float* dup,
                             double* lossp, int64_t* blocks_out, hipEvent_t start,
                             hipEvent_t stop, hipStream_t s);
// After the fused step: the repeated rows (short runs, pieces, and rows
// whose pieces are combined by the last piece to finish) and, with a loss
// output, the loss sum (the fused step's partials in a fixed order).
struct FinishArgs {
    int64_t m;               // occurrences of the batch (0: no records)
    const uint4* shorts;     // its short-run records (Control::nshort of them)
    const uint4* pieces;     // its pieces (Control::npiece)
    const uint4* combs;
    uint32_t* ccount;
    const float* dup;
    double* part;
    ListCaps caps;
    float lr;
    const double* lossp;   // per-workgroup loss partials of the fused step
    int64_t loss_blocks;   // how many
    double* loss_out;      // or null: no loss
};
// stop (if not null) is recorded by the kernel's own completion, not by a
// separate queue packet.
hipError_t launch_finish(const TableArgs& t, Control* ctl, const FinishArgs& f, hipEvent_t stop,
                         hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s);
hipError_t launch_walks(const WalkArgs& A, uint32_t* counts, uint64_t* offsets, int64_t* total,
                        int64_t capacity, int32_t* src, int32_t* dst, int32_t* cc, int32_t* hist,
                        int32_t* status, hipStream_t s);
// Per-positive weights from distance histograms (k_tables.hip)
constexpr int kMaxHistWindow = 32;
hipError_t launch_cocount_weights(const int32_t* hist, int64_t n, int window, const float* wd,
                                  float* out, hipStream_t s);
// Embedding evaluation (k_eval.hip)
hipError_t launch_eval_status_clear(int32_t* status, hipStream_t s);
hipError_t launch_eval_pairs(const int64_t* off, const int32_t* nbr, int64_t N, int64_t E,
                             uint64_t seed, int64_t n_edge, int64_t n_non, int32_t max_tries,
                             int32_t* u, int32_t* v, int32_t* status, hipStream_t s);
hipError_t launch_eval_dist(const float* T, int64_t N, int32_t D, const int32_t* u,
                            const int32_t* v, int64_t n, float* out, int32_t* status,
                            hipStream_t s);
constexpr int kEvalSumBlocks = 256;
hipError_t launch_eval_sums(const float* d, int64_t n_edge, int64_t n, double* part, double* out,
                            hipStream_t s);
hipError_t launch_eval_keys(const float* d, int64_t n, uint32_t* keys, hipStream_t s);
hipError_t launch_eval_quantiles(const uint32_t* sorted, const double* cnt, const double* q,
                                 int nq, double* out, hipStream_t s);
int knn_pass_queries(int D);
int64_t knn_lists(int64_t N, int D, int QB);
// Workspace of a nearest-row search (device memory, one pass of queries).
struct KnnBuffers {
    float* qn;        // [kKnnPass][dim] normalised queries
    float* qn2;       // [kKnnPass] their squared norms (0 or 1)
    int32_t* qid;     // [kKnnPass] their rows (-1: padding)
    uint64_t* partial;  // per-wave lists of the list-merging search
    float* tau;       // [kKnnPass] distance bound of the next threshold scan
    uint32_t* cnt;    // [kKnnPass] candidates of the current scan
    uint64_t* cand;   // [kKnnPass][kKnnCandCap] their keys
    int32_t* gate;    // 1: a final scan overflowed, the list-merging search runs
};
hipError_t launch_knn(const float* T, int64_t N, int32_t D, const int32_t* q, int32_t nq,
                      int32_t k, int32_t* ids, float* dist, const KnnBuffers& B,
                      bool lists_only, int32_t* status, hipStream_t s);
hipError_t launch_eval_recall(const int64_t* off, const int32_t* nbr, int64_t N, int64_t E,
                              const int32_t* q, int32_t nq, const int32_t* ids, int32_t k,
                              double* out, int32_t* status, hipStream_t s);
hipError_t launch_loss_final(Control* ctl, const double* lossp, int64_t blocks, double* out,
                             hipStream_t s);
hipError_t launch_atomic_gather(const TableArgs& t, Control* ctl, const StepArgs& a,
                                const int32_t* neg, float* gsrc, float* coef, double* lossp,
                                int64_t* blocks_out, hipStream_t s);
hipError_t launch_atomic_scatter_T(const TableArgs& t, Control* ctl, const StepArgs& a,
                                   const int32_t* neg, const float* coef, hipStream_t s);
hipError_t launch_atomic_scatter_S(const TableArgs& t, Control* ctl, const StepArgs& a,
                                   const float* gsrc, hipStream_t s);
hipError_t launch_eval(const TableArgs& t, Control* ctl, const StepArgs& a, double* lossp,
                       int64_t* blocks_out, hipStream_t s);

hipError_t launch_probe(const TableArgs& t, Control* ctl, const int32_t* src, const int32_t* dst,
                        int64_t n, uint64_t first_pos, hipStream_t s);


}  // namespace huge
