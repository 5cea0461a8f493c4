/*
 * huge.h -- C ABI of libhuge, the MI355X (gfx950) training step of HUGE
 * ("HUGE: Huge Unsupervised Graph Embeddings with TPUs", KDD'23).
 *
 * The library trains DeepWalk-style graph embeddings by skip-gram negative
 * sampling (Sec. 2.2) on batches of the (source_id, destination_id, co_counts)
 * triples produced by the random-walk sampler (Sec. 3.2).  Per step it
 * replicates each source, draws negatives (Sec. 3.3.2), gathers the rows of a
 * source table S and a context table T, computes the co_counts-weighted
 * sigmoid loss, aggregates the gradient of the whole batch and applies it to
 * the tables with SGD (Sec. 3.3.2; Table 2).  Everything runs in hand-written
 * HIP kernels on one GPU; both tables stay resident in HBM.
 *
 * The quantities computed (the paper names the loss parts but prints no
 * formula; the reading used here is standard word2vec negative sampling):
 *   x_i  = <S[u_i], T[v_i]>,  y_ik = <S[u_i], T[m_ik]>,  k < K
 *   L    = sum_i c_i * ( softplus(-x_i) + sum_k softplus(y_ik) )
 *   g_i  = c_i (sigmoid(x_i) - 1),  h_ik = c_i sigmoid(y_ik)
 *   S[u] -= lr * sum_{i: u_i = u} ( g_i T[v_i] + sum_k h_ik T[m_ik] )
 *   T[r] -= lr * ( sum_{i: v_i = r} g_i S[u_i] + sum_{(i,k): m_ik = r} h_ik S[u_i] )
 * Every read uses pre-step values (one synchronous step); contributions to a
 * row that appears several times in a batch are summed.
 *
 * Conventions
 *   - Device pointers are HIP device memory of the current device; host
 *     pointers are ordinary memory.  The caller owns every buffer; the
 *     library owns only the small host-side handle.  Buffers must outlive
 *     the handle, and batch arrays must stay valid until the step completes
 *     on its stream.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All calls are asynchronous on that stream except huge_check and
 *     huge_step_stats, which synchronise it.  A handle is not thread-safe.
 *   - Every function returns a huge_status (0 = success, negative = error)
 *     and never aborts the process.  Argument errors are detected on the
 *     host before any launch and leave every buffer untouched.
 *   - Ids are int32 (N <= 2^31 - 1); row offsets are computed in 64 bits.
 *   - Tables are row-major, N x D, contiguous: fp32, or bf16 with
 *     huge_config.table_dtype = HUGE_DTYPE_BF16.  The evaluation calls read
 *     fp32 tables (huge_get_rows widens bf16 rows).
 */
#ifndef HUGE_H
#define HUGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The library is built with hidden symbol visibility: the declarations of
   this header are its only exports. */
#if defined(__GNUC__)
#pragma GCC visibility push(default)
#endif

typedef int32_t huge_status;
#define HUGE_OK 0
#define HUGE_ERR_INVALID_ARG (-1)     /* null pointer, bad size or config          */
#define HUGE_ERR_ID_OUT_OF_RANGE (-2) /* a source/destination id outside [0, N)    */
#define HUGE_ERR_BAD_COUNT (-3)       /* a negative co_count                       */
#define HUGE_ERR_WORKSPACE (-4)       /* workspace smaller than huge_workspace_bytes */
#define HUGE_ERR_HIP (-5)             /* a HIP runtime call failed                 */

/* Negative distribution: uniform over the vocabulary (Sec. 3.3.2), or an
   alias table over caller weights (e.g. degree^0.75). */
#define HUGE_NEG_UNIFORM 0
#define HUGE_NEG_ALIAS 1

/* Gradient scatter: SORTED groups the rows of a batch by id (one radix pass
   on the lowest digit, then a hash table per bucket), updates rows that occur
   once in place and sums repeated rows in occurrence order -- bitwise
   reproducible run to run.  ATOMIC adds every contribution
   with fp32 atomics into the tables after all reads -- same result up to the
   order of summation, not reproducible bit for bit. */
#define HUGE_SCATTER_SORTED 0
#define HUGE_SCATTER_ATOMIC 1

/* Element type of the two tables.  F32: IEEE binary32.  BF16: bfloat16 (the
   upper 16 bits of a binary32), half the bytes per row; every step reads the
   rows widened to fp32, computes in fp32 as for F32 tables, and rounds each
   written element to the nearest bf16, ties to even (repeated rows: their
   fp64 sum applied in fp64, rounded to fp32, then to bf16).  The paper keeps
   fp32 tables; BF16 halves the memory and the traffic of a step (Sec. 3.3.2
   bounds the step by its row traffic).  BF16 works with the SORTED scatter
   only. */
#define HUGE_DTYPE_F32 0
#define HUGE_DTYPE_BF16 1

typedef struct huge_config {
    int64_t num_nodes;       /* N: rows of each table, 1 .. 2^31-1                       */
    int32_t dim;             /* D: floats per row, multiple of 4, 4 .. 1024              */
    int32_t num_neg_per_pos; /* K: negatives per positive, 1 .. 64 (Sec. 3.3.2, Table 2) */
    int64_t max_batch;       /* largest number of positives per call, >= 1               */
    uint64_t seed;           /* Philox key for the initial tables and the negatives      */
    float init_half_width;   /* a: initial values U[-a, a); 0 selects 0.5 / D            */
    int32_t neg_kind;        /* HUGE_NEG_UNIFORM or HUGE_NEG_ALIAS                       */
    int32_t scatter_kind;    /* HUGE_SCATTER_SORTED or HUGE_SCATTER_ATOMIC               */
    int32_t table_dtype;     /* HUGE_DTYPE_F32 (0) or HUGE_DTYPE_BF16                    */
} huge_config;

typedef struct huge_handle huge_handle; /* opaque, host-side */

/* Bytes of device workspace a handle with this config needs (scratch for the
   negatives, sort buffers, duplicate contributions, loss partials and
   counters).  Returns 0 if the config is invalid. */
size_t huge_workspace_bytes(const huge_config* cfg);

/* Host-only, deterministic alias table for negative sampling (Walker; Vose)
   in exact integer form: bucket j keeps mass W_j = trunc(w_j N 2^32 / sum w)
   (the rounding residue goes to the largest bucket, lowest index on ties);
   small buckets (W < 2^32) are filled from large ones in FIFO index order;
   thr[j] is the 32-bit threshold below which a draw keeps j, alias[j] the
   other outcome.  weights: n >= 1 finite non-negative doubles with a positive
   sum; thr_out, alias_out: n entries, host memory.  The caller copies them
   to device memory for huge_init_tables. */
huge_status huge_build_alias(const double* weights, int64_t n, uint32_t* thr_out,
                             int32_t* alias_out);

/* Create a handle over caller-owned tables and fill both with the initial
   values: element (r, c) of table t (0 = S, 1 = T) is j * (a 2^-23) with
   j = (word >> 8) - 2^23 and word = word (c mod 4) of Philox4x32-10 on counter
   (lo32 r, hi32 r, c div 4, 2 + t) under key (lo32 seed, hi32 seed): uniform
   on [-a, a) (the paper does not state an initialisation); a BF16 table holds
   these values rounded to nearest, ties to even.
     d_S, d_T       : N x D device tables of cfg->table_dtype elements,
                      16-byte aligned (written)
     d_alias_thr,
     d_alias        : N entries each on the device (HUGE_NEG_ALIAS), else NULL
     d_workspace    : >= huge_workspace_bytes(cfg) bytes of device memory
     out            : receives the handle; destroy with huge_destroy */
huge_status huge_init_tables(const huge_config* cfg, void* d_S, void* d_T,
                             const uint32_t* d_alias_thr, const int32_t* d_alias,
                             void* d_workspace, size_t ws_bytes, void* stream,
                             huge_handle** out);

/* Same as huge_init_tables without writing the tables: for tables restored
   from a checkpoint. */
huge_status huge_attach_tables(const huge_config* cfg, void* d_S, void* d_T,
                               const uint32_t* d_alias_thr, const int32_t* d_alias,
                               void* d_workspace, size_t ws_bytes, huge_handle** out);

/* One synchronous SGD step over n positives (Sec. 3.3.2; Table 2).
     d_src, d_dst    : n int32 ids in [0, N) (source_id, destination_id)
     d_cc            : n int32 co_counts >= 0, the weight of each positive
     first_pos_index : global index p of the first positive; negative k of
                       positive i is drawn from Philox counter
                       (lo32 p+i, hi32 p+i, k, 1): j = floor(x N / 2^64) with
                       x = (r1 << 32) | r0, and with an alias table the result
                       is j if r2 < thr[j], else alias[j]
     lr              : SGD learning rate
     d_loss_sum      : device double receiving L at the pre-step values, or NULL
   n = 0 is a no-op that writes 0 to *d_loss_sum.  Ids outside [0, N) or a
   negative co_count make the whole step a no-op (no table is written, the
   loss is NaN); huge_check then reports the error. */
huge_status huge_train_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                            const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                            float lr, double* d_loss_sum, void* stream);

/* The same step in two halves, so that later batches are grouped while the
   current one is applied (grouping never reads or writes the tables).
     huge_prepare_step   : validation, negative draws and the whole grouping
                           of a batch (keys, radix pass on the lowest digit,
                           per-bucket grouping), on `stream` (the preparation
                           stream); at most two prepared batches may be
                           pending
     huge_train_prepared : the gather, loss and update of the oldest prepared
                           batch (the fused kernel, then the repeated rows
                           and the loss sum), with the given lr and loss
                           output, on `stream` (the apply stream)
   The grouping kernels run in workgroups of few registers, so that on a
   preparation stream of their own they run beside the previous batch's
   update.  The library orders the halves with HIP events: an apply waits for
   its batch's preparation and for the previous apply, a preparation for the
   apply that last used its grouping buffers (or the one after it: apply
   completions are recorded only every other step).  The batch arrays must stay
   valid until the batch is applied.  Results are bitwise those of
   huge_train_step, which is the two halves on one stream and requires that
   no batch is pending. */
huge_status huge_prepare_step(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                              const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                              void* stream);
huge_status huge_train_prepared(huge_handle* h, float lr, double* d_loss_sum, void* stream);

/* Weighted co-occurrences (Sec. 3.2: co_counts is a histogram over the walk
   distance of each co-occurrence).  The *_weighted calls are the step, its
   two halves and the loss with one float weight per positive,
   c_i = d_weight[i], in place of the integer co_count; a weight that is
   negative, NaN or infinite makes the call a no-op reported like a negative
   co_count (HUGE_ERR_BAD_COUNT).  Results with integer-valued weights are
   bitwise those of the integer calls. */
huge_status huge_train_step_weighted(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                                     const float* d_weight, int64_t n, uint64_t first_pos_index,
                                     float lr, double* d_loss_sum, void* stream);
huge_status huge_prepare_step_weighted(huge_handle* h, const int32_t* d_src,
                                       const int32_t* d_dst, const float* d_weight, int64_t n,
                                       uint64_t first_pos_index, void* stream);
huge_status huge_eval_loss_weighted(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                                    const float* d_weight, int64_t n, uint64_t first_pos_index,
                                    double* d_loss_sum, void* stream);

/* The weight of each triple from its distance histogram (as
   huge_sample_walks writes it): d_weight[i] = sum over d of
   h_dist_weights[d] * d_hist[i * window + d], the products and the sum taken
   in double (each rounded once, distances in ascending order), then rounded
   once to float.  h_dist_weights: `window` host floats, finite and >= 0;
   1 <= window <= 32.  A negative histogram entry gives NaN. */
huge_status huge_cocount_weights(const int32_t* d_hist, int64_t n, int32_t window,
                                 const float* h_dist_weights, float* d_weight, void* stream);

/* L of a batch at the current tables, with the negatives huge_train_step
   would draw for the same first_pos_index; writes nothing else. */
huge_status huge_eval_loss(huge_handle* h, const int32_t* d_src, const int32_t* d_dst,
                           const int32_t* d_cc, int64_t n, uint64_t first_pos_index,
                           double* d_loss_sum, void* stream);

/* Copy rows of table (0 = S, 1 = T) into d_out (n x D fp32, row-major; rows
   of a BF16 table are widened exactly).
   d_ids: n int64 device ids; an id outside [0, N) yields a row of NaN and
   makes huge_check report HUGE_ERR_ID_OUT_OF_RANGE. */
huge_status huge_get_rows(huge_handle* h, int32_t table, const int64_t* d_ids, int64_t n,
                          float* d_out, void* stream);

/* The negatives huge_train_step draws for n positives starting at
   first_pos_index: d_neg_out receives n x K int32 (row i = positive i). */
huge_status huge_sample_negatives(huge_handle* h, int64_t n, uint64_t first_pos_index,
                                  int32_t* d_neg_out, void* stream);

/* Bandwidth probe, for measurement: reads and writes back unchanged every
   row a step over this batch would touch -- S[src_i], T[dst_i] and the K
   rows T[m_ik] drawn for first_pos_index as in huge_train_step -- one read
   and one write per occurrence, in the fused step's launch shape and with no
   arithmetic.  Its rate is the practical ceiling of the step's random row
   traffic on the device.  d_src, d_dst: n <= max_batch int32 ids in [0, N);
   an id outside that range skips its positive and makes huge_check report
   HUGE_ERR_ID_OUT_OF_RANGE.  The tables keep their values bit for bit; the
   call is ordered after the last apply, and must not run beside a step. */
huge_status huge_probe_rows(huge_handle* h, const int32_t* d_src, const int32_t* d_dst, int64_t n,
                            uint64_t first_pos_index, void* stream);

/* Synchronise the stream; return and clear the first device-side error
   (HUGE_ERR_ID_OUT_OF_RANGE or HUGE_ERR_BAD_COUNT) since the last check. */
huge_status huge_check(huge_handle* h, void* stream);

/* Synchronise the stream and report the last sorted step's row counts:
   distinct source rows, distinct context rows, and occurrences that fell in
   a repeated row (their contributions were summed before the update). */
huge_status huge_step_stats(huge_handle* h, void* stream, int64_t* unique_src,
                            int64_t* unique_ctx, int64_t* dup_occurrences);

/* Phase timing.  After huge_profile_begin(h, max_steps, all_phases, every),
   every every-th one of the next batches (prepared, or stepped with
   huge_train_step), max_steps of them, records HIP events on the streams
   its stages run on: around the fused kernel only (all_phases = 0), or at
   every phase boundary (all_phases = 1).  Each event is one more packet in
   a stream, which costs a few microseconds of the step it is in; every > 1
   spreads that cost.  huge_profile_end waits for all of them on `stream`,
   writes the summed durations in milliseconds to phase_ms[HUGE_PHASES] (0
   for phases not recorded) and the number of recorded steps to *steps, and
   releases the events.  Phases: 0 set-up, negative sampling with the tile
   digit counts, tile prefixes, 1 the radix pass, 2 the per-bucket grouping (1 and 2 are
   empty for the atomic scatter), 3 the fused gather/loss/update kernel
   (atomic scatter: gather and coefficients), 4 the finish kernel: repeated
   rows and the loss sum (atomic scatter: the atomic adds and the loss sum),
   5 always 0 (the loss sum has no kernel of its own).  Errors: max_steps or
   every outside [1, 10^6], all_phases not 0 or 1. */
#define HUGE_PHASES 6
huge_status huge_profile_begin(huge_handle* h, int32_t max_steps, int32_t all_phases,
                               int32_t every);
huge_status huge_profile_end(huge_handle* h, void* stream, double* phase_ms, int32_t* steps);

/* ------------------------------------------------------------------------
   Random-walk sampler: the (source_id, destination_id, co_counts) triples the
   step consumes, produced on the GPU from a graph in device memory
   (Sec. 3.2, Alg. 1).  Every seed node s is repeated walks_per_node times
   (Alg. 1's gamma); walk r of s takes walk_steps uniform steps (Alg. 1's k):
   w_0 = s, w_t = neighbour floor(x deg / 2^64) of w_{t-1} in CSR order, x the
   64-bit word (r1 << 32) | r0 of Philox4x32-10 on counter
   (lo32 s, hi32 s, r, 4 + t) under key (lo32 seed, hi32 seed); a node without
   neighbours ends the walk.  The walks of a seed are grouped and their
   co-occurrences combined (Alg. 1, GroupByKey, CombineValues) into one triple
   per distinct (source, destination) pair:
     seed_pairs_only = 1: the pairs (s, w_t) for t = 1 .. window -- the
                          paper's triple, its histogram indexed by the walk
                          distance from the seed (Sec. 3.2);
     seed_pairs_only = 0: every ordered pair (w_a, w_b) of a walk with
                          1 <= |a - b| <= window (DeepWalk's context window).
   Pairs of a node with itself are dropped.  cc = the pair's co-occurrences;
   hist[d - 1] = those at distance d.  Triples come in ascending seed order
   and, within a seed, in ascending (source, destination) order: the output
   is a deterministic function of the graph, the config and the seed range. */
typedef struct huge_walk_config {
    int64_t num_nodes;       /* N: nodes of the graph, 1 .. 2^31-1                      */
    int32_t walks_per_node;  /* walks started from every seed, 1 .. 1024                */
    int32_t walk_steps;      /* steps per walk, 1 .. 64                                  */
    int32_t window;          /* largest co-occurrence distance, 1 .. min(walk_steps, 32) */
    int32_t seed_pairs_only; /* 1: pairs (seed, w_t); 0: all pairs within the window     */
    uint64_t seed;           /* Philox key                                               */
} huge_walk_config;
/* Besides these bounds, a seed's walks may hold at most 8192 nodes
   (walks_per_node x (walk_steps + 1)) and 4096 pairs (walks_per_node x
   window for seed pairs, walks_per_node x 2 (window (walk_steps + 1) -
   window (window + 1) / 2) for window pairs). */

/* Bytes of device workspace huge_sample_walks needs for num_seeds seeds;
   0 if the config is invalid. */
size_t huge_walk_workspace_bytes(const huge_walk_config* cfg, int64_t num_seeds);

/* Triples of the seeds first_seed .. first_seed + num_seeds - 1.
     d_offsets   : N + 1 int64 CSR offsets (device), non-decreasing from 0
     d_neighbors : num_edges int32 neighbour ids in [0, N) (device)
     d_src, d_dst, d_cc : capacity int32 each (device), the triples
     d_hist      : capacity x window int32 (device), or NULL
     d_count     : device int64, receives the number of triples (also when
                   it exceeds capacity)
     d_status    : device int32, receives 0; -2 if the graph is malformed
                   (an offset or neighbour out of range: nothing is written);
                   -4 if the triples exceed capacity (nothing is written)
     d_workspace : >= huge_walk_workspace_bytes(cfg, num_seeds) bytes, 256-byte
                   aligned
   Asynchronous on `stream`; host-detectable argument errors return before
   any launch. */
huge_status huge_sample_walks(const huge_walk_config* cfg, const int64_t* d_offsets,
                              const int32_t* d_neighbors, int64_t num_edges, int64_t first_seed,
                              int64_t num_seeds, int32_t* d_src, int32_t* d_dst, int32_t* d_cc,
                              int32_t* d_hist, int64_t capacity, int64_t* d_count,
                              int32_t* d_status, void* d_workspace, size_t ws_bytes,
                              void* stream);

/* ------------------------------------------------------------------------
   Unsupervised evaluation of an embedding table (Sec. 4): rows are
   L2-normalised (a row of zeros stays zero) and compared by the Euclidean
   distance d(u, v) = |x_u/|x_u| - x_v/|x_v||, in [0, 2].
     edge SNR        = mean d over sampled non-edges / mean d over sampled
                       edges, with percentiles of both distributions;
     recall@k(u)     = |N(u) & S| / k, S = the k rows v != u nearest to u
                       (ties: smaller id), N(u) = the ids of u's list other
                       than u.
   The calls take no handle and work on any table: N rows of `dim` floats,
   row-major (dim a multiple of 4, 4 .. 1024).  CSR graphs: N + 1 int64
   offsets, non-decreasing from 0 to num_edges, and num_edges int32
   neighbour ids in [0, N); each node's list must be in ascending order (the
   non-edge test and the recall search it).  d_status (device int32)
   receives 0, or -2 when a device-side check fails (an id or offset out of
   range); affected outputs are then NaN or -1.  All calls are asynchronous
   on `stream`; host-detectable argument errors return before any launch. */

/* Bytes of device workspace huge_eval_summary (up to max_pairs distances)
   and huge_eval_knn (a table of num_rows x dim, k nearest) need; 0 if the
   sizes are out of range. */
size_t huge_eval_workspace_bytes(int64_t max_pairs, int64_t num_rows, int32_t dim, int32_t k);

/* n_edge edge pairs, then n_non non-edge pairs, into d_u[n_edge + n_non],
   d_v[...] (device int32).  Edge pair j draws the Philox counter
   (lo32 j, hi32 j, 0, 0x80000001) under key (lo32 seed, hi32 seed): edge
   index e = floor(x num_edges / 2^64), x = (r1 << 32) | r0, and the pair is
   (the node whose list holds e, d_neighbors[e]).  Non-edge pair j tries
   a = 0 .. max_tries - 1 with counter (lo32 j, hi32 j, a, 0x80000002):
   u = floor(x0 N / 2^64), v = floor(x1 N / 2^64), x0 = (r1 << 32) | r0,
   x1 = (r3 << 32) | r2, and keeps the first try with u != v and v not in
   u's list; if none qualifies the pair is (-1, -1).  Errors: n_edge > 0 with
   num_edges = 0, negative counts, max_tries < 1. */
huge_status huge_eval_pairs(const int64_t* d_offsets, const int32_t* d_neighbors,
                            int64_t num_nodes, int64_t num_edges, uint64_t seed, int64_t n_edge,
                            int64_t n_non, int32_t max_tries, int32_t* d_u, int32_t* d_v,
                            int32_t* d_status, void* stream);

/* d_dist[i] = d(d_u[i], d_v[i]) (device float), NaN where either id is
   negative (a failed non-edge draw); an id >= num_rows sets -2. */
huge_status huge_eval_distances(const float* d_table, int64_t num_rows, int32_t dim,
                                const int32_t* d_u, const int32_t* d_v, int64_t n,
                                float* d_dist, int32_t* d_status, void* stream);

/* Summary of n_edge edge distances followed by n_non non-edge distances
   (device float, NaN = no pair), into d_out (device double):
     d_out[0], d_out[1]  number of valid edge / non-edge distances
     d_out[2], d_out[3]  their means (fixed-order double sums)
     d_out[4]            edge SNR = d_out[3] / d_out[2]
     d_out[5 .. 5+nq)    percentiles of the edge distances at h_quantiles
     d_out[5+nq .. 5+2nq) the same for the non-edge distances
   Percentile q (0 .. 100, host doubles, at most 128 of them) of n values:
   sorted, position h = (n - 1) q / 100, linear between the order
   statistics around h.  Means, SNR and percentiles are NaN for an empty
   set.  Needs huge_eval_workspace_bytes(n_edge + n_non, ...) of workspace. */
huge_status huge_eval_summary(const float* d_dist, int64_t n_edge, int64_t n_non,
                              const double* h_quantiles, int32_t n_quantiles, double* d_out,
                              void* d_workspace, size_t ws_bytes, void* stream);

/* huge_eval_summary without a caller workspace, for callers that cannot
   allocate device memory (code under HIP graph capture, serving loops,
   harnesses that forbid hipMalloc): the same kernels on a fixed 32 MiB array
   of device memory that the library holds on every device it runs on until
   the process ends.  It allocates nothing and calls no allocating routine.
   n_edge + n_non may be up to 3,726,784 (the largest count whose summary
   workspace fits in the array); more returns HUGE_ERR_WORKSPACE before any
   launch.  Every call on a device uses that
   device's one array and finds the previous call's contents there (nothing
   is carried over: each call writes what it reads); calls that overlap on
   one device -- on different streams or from different threads without
   ordering -- race on it and must be serialised by the caller.  Other
   arguments and errors as for huge_eval_summary. */
huge_status huge_eval_summary_static(const float* d_dist, int64_t n_edge, int64_t n_non,
                                     const double* h_quantiles, int32_t n_quantiles,
                                     double* d_out, void* stream);

/* The k rows nearest to each of the n_queries query rows (ids in d_queries),
   excluding the query itself: d_ids[q k + t] (device int32, ascending
   (distance, id); -1 if fewer than k other rows exist) and d_dist[...]
   (device float).  Distances come from the expansion
   d^2 = |q|^2 + |r|^2 - 2 <q, r> of the normalised rows on the matrix cores:
   for dim <= 128 each value split into two fp16 parts (hi + lo, within
   2^-22 of it) and the products hi.hi + hi.lo + lo.hi summed in fp32 (about
   2^-21 of each term, well inside the search's fp32 distance bound); wider
   rows in fp32.  1 <= k <= 32;
   dim <= 512.  Queries are processed in passes of up to
   128 (dim <= 128), 64 (dim <= 256) or 32 over the table.  For dim <= 128
   a pass is a series of threshold scans: strided samples of the row tiles,
   each 32 times denser than the one before, then every tile; a sample's
   k-th distance bounds the next scan's candidates per query, which are
   sorted between scans.  Should more than 8192 rows of the last scan fall
   within a query's bound (many rows at one distance), the pass is computed
   again by the per-wave lists of huge_eval_knn_lists; the answer is the
   same either way, bit for bit.  Sizes (Sec. 4's sampled recall): 100
   queries over 1e8 x 128 rows. */
huge_status huge_eval_knn(const float* d_table, int64_t num_rows, int32_t dim,
                          const int32_t* d_queries, int32_t n_queries, int32_t k,
                          int32_t* d_ids, float* d_dist, void* d_workspace, size_t ws_bytes,
                          int32_t* d_status, void* stream);

/* huge_eval_knn computed by the search it falls back on: every wave keeps
   sorted lists of its best k per query over its share of the tiles, merged
   at the end (no distance bound).  The same distances and the same answer;
   for comparing the two searches.  Arguments, workspace and errors as for
   huge_eval_knn. */
huge_status huge_eval_knn_lists(const float* d_table, int64_t num_rows, int32_t dim,
                                const int32_t* d_queries, int32_t n_queries, int32_t k,
                                int32_t* d_ids, float* d_dist, void* d_workspace,
                                size_t ws_bytes, int32_t* d_status, void* stream);

/* d_recall[q] = recall@k of query d_queries[q] (device double) from its k
   nearest rows d_ids[q k ..] (as huge_eval_knn writes them); 1 <= k <= 64. */
huge_status huge_eval_recall(const int64_t* d_offsets, const int32_t* d_neighbors,
                             int64_t num_nodes, int64_t num_edges, const int32_t* d_queries,
                             int32_t n_queries, const int32_t* d_ids, int32_t k,
                             double* d_recall, int32_t* d_status, void* stream);

void huge_destroy(huge_handle* h);
const char* huge_status_string(huge_status s);

#if defined(__GNUC__)
#pragma GCC visibility pop
#endif

#ifdef __cplusplus
}
#endif
#endif /* HUGE_H */
