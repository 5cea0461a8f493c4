/*
 * huge_oracle.c -- CPU oracle for the HUGE embedding training step.
 *
 * TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load this file.  It shares no code,
 * header, table or constant generator with the GPU library; both sides are
 * written independently from the same published definitions.
 *
 * What it computes (HUGE, KDD'23, arXiv 2307.14490):
 *   - DeepWalk trained as word2vec with negative sampling (Sec. 2.2): each
 *     co-occurrence (source_id, destination_id, co_counts) (Sec. 3.2, the
 *     sampler's output triple) is a "positive" example; the source id is
 *     replicated and num_neg_per_pos destination ids are drawn as "negative"
 *     examples (Sec. 3.3.2); the loss has a positive and a negative part
 *     (Sec. 3.2).
 *   - one synchronous step: gradients of the whole batch are aggregated and
 *     then applied to the embedding tables (Sec. 3.3.2), plain SGD (Table 2).
 *
 * Readings of points the paper leaves open (listed in the design notes):
 *   loss       L = sum_i c_i [ softplus(-x_i) + sum_k softplus(y_ik) ]
 *              x_i = <S[u_i], T[v_i]>,  y_ik = <S[u_i], T[m_ik]>
 *              (co_counts c_i weighs the whole term; the batch loss is a sum)
 *   gradient   g_i = c_i (sigma(x_i) - 1),  h_ik = c_i sigma(y_ik)
 *              dS[u_i] += g_i T[v_i] + sum_k h_ik T[m_ik]
 *              dT[v_i] += g_i S[u_i],  dT[m_ik] += h_ik S[u_i]
 *   update     every read uses pre-step values; contributions to a row that
 *              occurs several times are summed; row <- row - lr * grad.
 *   negatives  drawn with replacement, no rejection, from a counter-based
 *              Philox4x32-10 stream (Salmon et al., SC'11): uniform over
 *              [0, N) or through a Walker/Vose alias table over given weights.
 *   init       both tables U[-a, a) from the same Philox stream.
 *
 * Precision: gradients, dots and the loss in double; tables are float32
 * (the storage type), each touched element is rounded once when the step is
 * applied.  Accumulation order per row: positive index ascending, then the
 * destination slot, then negatives in slot order.
 *
 * Plain C99, single-threaded, no SIMD, no blocking.  Error codes:
 *   0 ok, -1 invalid argument, -2 id out of range, -3 negative co_count.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_OK 0
#define OR_EINVAL (-1)
#define OR_ERANGE (-2)
#define OR_ECOUNT (-3)

/* ------------------------------------------------------------------------- */
/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As   */
/* Easy as 1, 2, 3", SC'11): 10 rounds of the 4x32 Philox S-box with the     */
/* published multipliers and Weyl key increments.                            */
/* ------------------------------------------------------------------------- */
void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2],
                          uint32_t out[4]) {
    const uint32_t mult0 = 0xD2511F53u, mult1 = 0xCD9E8D57u;
    const uint32_t weyl0 = 0x9E3779B9u, weyl1 = 0xBB67AE85u;
    uint32_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += weyl0;
            k1 += weyl1;
        }
        uint64_t prod0 = (uint64_t)mult0 * (uint64_t)x0;
        uint64_t prod1 = (uint64_t)mult1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(prod0 >> 32), lo0 = (uint32_t)prod0;
        uint32_t hi1 = (uint32_t)(prod1 >> 32), lo1 = (uint32_t)prod1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

static void seed_key(uint64_t seed, uint32_t key[2]) {
    key[0] = (uint32_t)(seed & 0xFFFFFFFFu);
    key[1] = (uint32_t)(seed >> 32);
}

/* ------------------------------------------------------------------------- */
/* Table initialisation: U[-a, a).  Element (row, col) of table t (0 = source */
/* table S, 1 = context table T) takes word (col mod 4) of Philox block       */
/* counter (lo32(row), hi32(row), col div 4, 2 + t).  The top 24 bits of the  */
/* word give an integer j in [-2^23, 2^23) and the value is j * (a * 2^-23),  */
/* one float multiply.                                                        */
/* ------------------------------------------------------------------------- */
float oracle_init_value(uint64_t seed, int32_t table, int64_t row, int32_t col,
                        float half_width) {
    uint32_t key[2], ctr[4], out[4];
    seed_key(seed, key);
    ctr[0] = (uint32_t)((uint64_t)row & 0xFFFFFFFFu);
    ctr[1] = (uint32_t)((uint64_t)row >> 32);
    ctr[2] = (uint32_t)(col / 4);
    ctr[3] = (uint32_t)(2 + table);
    oracle_philox4x32_10(ctr, key, out);
    uint32_t word = out[col % 4];
    int32_t j = (int32_t)(word >> 8) - 8388608; /* 2^23 */
    float scale = (float)ldexp((double)half_width, -23);
    float v = (float)j * scale;
    return v;
}

/* Whole rows: one Philox block serves the four columns 4q .. 4q+3. */
int oracle_init_rows(uint64_t seed, int32_t table, const int64_t *rows, int64_t nrows,
                     int32_t dim, float half_width, float *out) {
    if (nrows < 0 || dim <= 0 || (nrows > 0 && (!rows || !out))) return OR_EINVAL;
    uint32_t key[2], ctr[4], word[4];
    seed_key(seed, key);
    float scale = (float)ldexp((double)half_width, -23);
    for (int64_t r = 0; r < nrows; ++r) {
        for (int32_t q = 0; 4 * q < dim; ++q) {
            ctr[0] = (uint32_t)((uint64_t)rows[r] & 0xFFFFFFFFu);
            ctr[1] = (uint32_t)((uint64_t)rows[r] >> 32);
            ctr[2] = (uint32_t)q;
            ctr[3] = (uint32_t)(2 + table);
            oracle_philox4x32_10(ctr, key, word);
            for (int32_t w = 0; w < 4 && 4 * q + w < dim; ++w) {
                int32_t j = (int32_t)(word[w] >> 8) - 8388608;
                out[r * dim + 4 * q + w] = (float)j * scale;
            }
        }
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Alias table (Walker 1977; Vose 1991) in exact integer form.               */
/*   1. total = sum of weights in double, ascending index order;             */
/*   2. W_j = trunc(w_j * (N * 2^32 / total)) as u64, the rounding residue    */
/*      (positive or negative) is added to the largest W (lowest index on    */
/*      ties), so that sum W_j == N * 2^32 exactly;                          */
/*   3. small = {j : W_j < 2^32}, large = the rest, FIFO in index order;      */
/*   4. while both are non-empty: s = pop(small), l = front(large);          */
/*      thr[s] = W_s, alias[s] = l, W_l -= 2^32 - W_s; if W_l < 2^32 then l   */
/*      moves from the front of large to the back of small;                   */
/*   5. every bucket left over keeps thr = 0xFFFFFFFF, alias = itself.        */
/* A draw picks a bucket j uniformly and a 32-bit coin r: j if r < thr[j],   */
/* alias[j] otherwise.                                                        */
/* ------------------------------------------------------------------------- */
int oracle_build_alias(const double *weights, int64_t n, uint32_t *thr, int32_t *alias) {
    if (n <= 0 || n > 2147483647LL || !weights || !thr || !alias) return OR_EINVAL;
    double total = 0.0;
    for (int64_t j = 0; j < n; ++j) {
        if (!(weights[j] >= 0.0) || isinf(weights[j])) return OR_EINVAL;
        total += weights[j];
    }
    if (!(total > 0.0) || isinf(total)) return OR_EINVAL;
    const uint64_t one = 4294967296ULL; /* 2^32 */
    uint64_t *W = (uint64_t *)malloc((size_t)n * sizeof(uint64_t));
    int64_t *small = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    int64_t *large = (int64_t *)malloc((size_t)n * sizeof(int64_t));
    if (!W || !small || !large) {
        free(W); free(small); free(large);
        return OR_EINVAL;
    }
    double scale = (double)n * 4294967296.0 / total;
    uint64_t sumW = 0;
    int64_t biggest = 0;
    for (int64_t j = 0; j < n; ++j) {
        W[j] = (uint64_t)(weights[j] * scale);
        sumW += W[j];
        if (W[j] > W[biggest]) biggest = j;
    }
    int64_t residue = (int64_t)((uint64_t)n * one - sumW);
    W[biggest] = (uint64_t)((int64_t)W[biggest] + residue);

    int64_t s_head = 0, s_tail = 0, l_head = 0, l_tail = 0;
    for (int64_t j = 0; j < n; ++j) {
        thr[j] = 0xFFFFFFFFu;
        alias[j] = (int32_t)j;
        if (W[j] < one) small[s_tail++] = j;
        else large[l_tail++] = j;
    }
    /* small is a FIFO over an array of n slots: every index enters it at most
       once, so s_tail never exceeds n. */
    while (s_head < s_tail && l_head < l_tail) {
        int64_t s = small[s_head++];
        int64_t l = large[l_head];
        thr[s] = (uint32_t)W[s];
        alias[s] = (int32_t)l;
        W[l] -= one - W[s];
        if (W[l] < one) {
            l_head++;
            small[s_tail++] = l;
        }
    }
    free(W); free(small); free(large);
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Negative sampling.  Negative k of the positive with global index p uses   */
/* Philox counter (lo32(p), hi32(p), k, 1) under key (lo32(seed), hi32(seed)).*/
/* The 64-bit word x = (r1 << 32) | r0 selects bucket floor(x * N / 2^64);    */
/* with an alias table, r2 is the coin.                                       */
/* ------------------------------------------------------------------------- */
int64_t oracle_sample_negative(uint64_t seed, uint64_t p, int32_t k, int64_t num_nodes,
                               const uint32_t *thr, const int32_t *alias) {
    uint32_t key[2], ctr[4], r[4];
    seed_key(seed, key);
    ctr[0] = (uint32_t)(p & 0xFFFFFFFFu);
    ctr[1] = (uint32_t)(p >> 32);
    ctr[2] = (uint32_t)k;
    ctr[3] = 1u;
    oracle_philox4x32_10(ctr, key, r);
    uint64_t x = ((uint64_t)r[1] << 32) | (uint64_t)r[0];
    unsigned __int128 wide = (unsigned __int128)x * (unsigned __int128)(uint64_t)num_nodes;
    int64_t j = (int64_t)(uint64_t)(wide >> 64);
    if (thr && alias) {
        if (!(r[2] < thr[j])) j = alias[j];
    }
    return j;
}

int oracle_sample_negatives(uint64_t seed, uint64_t first_pos, int64_t n, int32_t num_neg,
                            int64_t num_nodes, const uint32_t *thr, const int32_t *alias,
                            int32_t *neg_out) {
    if (n < 0 || num_neg < 1 || num_nodes < 1 || (n > 0 && !neg_out)) return OR_EINVAL;
    for (int64_t i = 0; i < n; ++i)
        for (int32_t k = 0; k < num_neg; ++k)
            neg_out[i * num_neg + k] = (int32_t)oracle_sample_negative(
                seed, first_pos + (uint64_t)i, k, num_nodes, thr, alias);
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Loss pieces, in double.                                                    */
/* ------------------------------------------------------------------------- */
static double sigmoid(double z) { return 1.0 / (1.0 + exp(-z)); }
static double softplus(double z) { return (z > 0.0 ? z : 0.0) + log1p(exp(-fabs(z))); }

/* The weight c_i of positive i: the float weight wf[i] where weights are
   given (a co-occurrence histogram combined with per-distance weights), else
   the integer co_count cc[i]. */
static double weight_of(const int32_t *cc, const float *wf, int64_t i) {
    return wf ? (double)wf[i] : (double)cc[i];
}

static int check_batch(int64_t ns, int64_t nt, int64_t n, int32_t num_neg,
                       const int32_t *src, const int32_t *dst, const int32_t *cc,
                       const float *wf, const int32_t *neg) {
    for (int64_t i = 0; i < n; ++i) {
        if (src[i] < 0 || src[i] >= ns || dst[i] < 0 || dst[i] >= nt) return OR_ERANGE;
        for (int32_t k = 0; k < num_neg; ++k) {
            int32_t m = neg[i * num_neg + k];
            if (m < 0 || m >= nt) return OR_ERANGE;
        }
    }
    for (int64_t i = 0; i < n; ++i) {
        if (wf) {
            if (!(wf[i] >= 0.0f && wf[i] <= 3.4028234663852886e38f)) return OR_ECOUNT;
        } else if (cc[i] < 0) {
            return OR_ECOUNT;
        }
    }
    return OR_OK;
}

static double dot_dd(const double *a, const double *b, int32_t dim) {
    double s = 0.0;
    for (int32_t d = 0; d < dim; ++d) s += a[d] * b[d];
    return s;
}

/*
 * Loss and gradient of the batch on double tables S (ns x dim) and T (nt x dim).
 * grad_S and grad_T (same shapes) are overwritten.  Returns 0 and writes the
 * loss, or an error code.
 */
static int sgns_grad_d(const double *S, const double *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const int32_t *cc, const float *wf, const int32_t *neg, double *grad_S,
                       double *grad_T, double *loss_out) {
    if (dim <= 0 || n < 0 || num_neg < 1 || !grad_S || !grad_T || !loss_out) return OR_EINVAL;
    int rc = check_batch(ns, nt, n, num_neg, src, dst, cc, wf, neg);
    if (rc) return rc;
    memset(grad_S, 0, (size_t)ns * (size_t)dim * sizeof(double));
    memset(grad_T, 0, (size_t)nt * (size_t)dim * sizeof(double));
    double loss = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double c = weight_of(cc, wf, i);
        const double *su = S + (int64_t)src[i] * dim;
        const double *tv = T + (int64_t)dst[i] * dim;
        double *gsu = grad_S + (int64_t)src[i] * dim;
        /* positive part */
        double x = dot_dd(su, tv, dim);
        double g = c * (sigmoid(x) - 1.0);
        loss += c * softplus(-x);
        double *gtv = grad_T + (int64_t)dst[i] * dim;
        for (int32_t d = 0; d < dim; ++d) {
            gsu[d] += g * tv[d];
            gtv[d] += g * su[d];
        }
        /* negative part */
        for (int32_t k = 0; k < num_neg; ++k) {
            int32_t m = neg[i * num_neg + k];
            const double *tm = T + (int64_t)m * dim;
            double *gtm = grad_T + (int64_t)m * dim;
            double y = dot_dd(su, tm, dim);
            double h = c * sigmoid(y);
            loss += c * softplus(y);
            for (int32_t d = 0; d < dim; ++d) {
                gsu[d] += h * tm[d];
                gtm[d] += h * su[d];
            }
        }
    }
    *loss_out = loss;
    return OR_OK;
}

int oracle_sgns_grad_d(const double *S, const double *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const int32_t *cc, const int32_t *neg, double *grad_S, double *grad_T,
                       double *loss_out) {
    if (n > 0 && !cc) return OR_EINVAL;
    return sgns_grad_d(S, T, ns, nt, dim, n, num_neg, src, dst, cc, NULL, neg, grad_S, grad_T,
                       loss_out);
}

/* Loss only, on double tables. */
int oracle_sgns_loss_d(const double *S, const double *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const int32_t *cc, const int32_t *neg, double *loss_out) {
    if (dim <= 0 || n < 0 || num_neg < 1 || !loss_out) return OR_EINVAL;
    int rc = check_batch(ns, nt, n, num_neg, src, dst, cc, NULL, neg);
    if (rc) return rc;
    double loss = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double c = (double)cc[i];
        const double *su = S + (int64_t)src[i] * dim;
        loss += c * softplus(-dot_dd(su, T + (int64_t)dst[i] * dim, dim));
        for (int32_t k = 0; k < num_neg; ++k)
            loss += c * softplus(dot_dd(su, T + (int64_t)neg[i * num_neg + k] * dim, dim));
    }
    *loss_out = loss;
    return OR_OK;
}

/*
 * One synchronous SGD step on float32 tables, in place.
 *   S: ns x dim, T: nt x dim (row-major); src/dst/cc: n entries;
 *   neg: n x num_neg negatives (from oracle_sample_negatives or a test);
 * The tables are widened to double, the gradient is taken at the pre-step
 * values, and each touched row is rewritten once as
 *   row = (float)((double)row - (double)lr * grad).
 * Rows that no example touches are not written.  On error nothing is written.
 */
static int sgns_step(float *S, float *T, int64_t ns, int64_t nt, int32_t dim, int64_t n,
                     int32_t num_neg, const int32_t *src, const int32_t *dst, const int32_t *cc,
                     const float *wf, const int32_t *neg, float lr, double *loss_out) {
    if (!S || !T || dim <= 0 || n < 0 || num_neg < 1 || !loss_out) return OR_EINVAL;
    if (n > 0 && (!src || !dst || (!cc && !wf) || !neg)) return OR_EINVAL;
    int rc = check_batch(ns, nt, n, num_neg, src, dst, cc, wf, neg);
    if (rc) return rc;
    size_t s_elems = (size_t)ns * (size_t)dim, t_elems = (size_t)nt * (size_t)dim;
    double *Sd = (double *)malloc(s_elems * sizeof(double));
    double *Td = (double *)malloc(t_elems * sizeof(double));
    double *gS = (double *)malloc(s_elems * sizeof(double));
    double *gT = (double *)malloc(t_elems * sizeof(double));
    unsigned char *touched_S = (unsigned char *)calloc((size_t)ns, 1);
    unsigned char *touched_T = (unsigned char *)calloc((size_t)nt, 1);
    if (!Sd || !Td || !gS || !gT || !touched_S || !touched_T) {
        free(Sd); free(Td); free(gS); free(gT); free(touched_S); free(touched_T);
        return OR_EINVAL;
    }
    for (size_t e = 0; e < s_elems; ++e) Sd[e] = (double)S[e];
    for (size_t e = 0; e < t_elems; ++e) Td[e] = (double)T[e];
    double loss = 0.0;
    rc = sgns_grad_d(Sd, Td, ns, nt, dim, n, num_neg, src, dst, cc, wf, neg, gS, gT, &loss);
    if (rc == OR_OK) {
        for (int64_t i = 0; i < n; ++i) {
            touched_S[src[i]] = 1;
            touched_T[dst[i]] = 1;
            for (int32_t k = 0; k < num_neg; ++k) touched_T[neg[i * num_neg + k]] = 1;
        }
        const double lr_d = (double)lr;
        for (int64_t r = 0; r < ns; ++r)
            if (touched_S[r])
                for (int32_t d = 0; d < dim; ++d)
                    S[r * dim + d] = (float)(Sd[r * dim + d] - lr_d * gS[r * dim + d]);
        for (int64_t r = 0; r < nt; ++r)
            if (touched_T[r])
                for (int32_t d = 0; d < dim; ++d)
                    T[r * dim + d] = (float)(Td[r * dim + d] - lr_d * gT[r * dim + d]);
        *loss_out = loss;
    }
    free(Sd); free(Td); free(gS); free(gT); free(touched_S); free(touched_T);
    return rc;
}

int oracle_sgns_step(float *S, float *T, int64_t ns, int64_t nt, int32_t dim, int64_t n,
                     int32_t num_neg, const int32_t *src, const int32_t *dst, const int32_t *cc,
                     const int32_t *neg, float lr, double *loss_out) {
    if (n > 0 && !cc) return OR_EINVAL;
    return sgns_step(S, T, ns, nt, dim, n, num_neg, src, dst, cc, NULL, neg, lr, loss_out);
}

/* The same step with a float weight per positive in place of the co_count
   (finite and >= 0, else OR_ECOUNT). */
int oracle_sgns_step_w(float *S, float *T, int64_t ns, int64_t nt, int32_t dim, int64_t n,
                       int32_t num_neg, const int32_t *src, const int32_t *dst, const float *w,
                       const int32_t *neg, float lr, double *loss_out) {
    if (n > 0 && !w) return OR_EINVAL;
    return sgns_step(S, T, ns, nt, dim, n, num_neg, src, dst, NULL, w, neg, lr, loss_out);
}

/* Loss of a batch on float32 tables, evaluated in double. */
static int sgns_loss(const float *S, const float *T, int64_t ns, int64_t nt, int32_t dim,
                     int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                     const int32_t *cc, const float *wf, const int32_t *neg, double *loss_out) {
    if (!S || !T || dim <= 0 || n < 0 || num_neg < 1 || !loss_out) return OR_EINVAL;
    if (n > 0 && !cc && !wf) return OR_EINVAL;
    int rc = check_batch(ns, nt, n, num_neg, src, dst, cc, wf, neg);
    if (rc) return rc;
    double *su = (double *)malloc((size_t)dim * sizeof(double));
    double *tr = (double *)malloc((size_t)dim * sizeof(double));
    if (!su || !tr) { free(su); free(tr); return OR_EINVAL; }
    double loss = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const double c = weight_of(cc, wf, i);
        for (int32_t d = 0; d < dim; ++d) su[d] = (double)S[(int64_t)src[i] * dim + d];
        for (int32_t d = 0; d < dim; ++d) tr[d] = (double)T[(int64_t)dst[i] * dim + d];
        loss += c * softplus(-dot_dd(su, tr, dim));
        for (int32_t k = 0; k < num_neg; ++k) {
            int64_t m = neg[i * num_neg + k];
            for (int32_t d = 0; d < dim; ++d) tr[d] = (double)T[m * dim + d];
            loss += c * softplus(dot_dd(su, tr, dim));
        }
    }
    free(su); free(tr);
    *loss_out = loss;
    return OR_OK;
}

int oracle_sgns_loss(const float *S, const float *T, int64_t ns, int64_t nt, int32_t dim,
                     int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                     const int32_t *cc, const int32_t *neg, double *loss_out) {
    return sgns_loss(S, T, ns, nt, dim, n, num_neg, src, dst, cc, NULL, neg, loss_out);
}

int oracle_sgns_loss_w(const float *S, const float *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const float *w, const int32_t *neg, double *loss_out) {
    return sgns_loss(S, T, ns, nt, dim, n, num_neg, src, dst, NULL, w, neg, loss_out);
}

/* ------------------------------------------------------------------------- */
/* Weights from distance histograms (Sec. 3.2: co_counts is a histogram over  */
/* the walk distance of a co-occurrence): positive i with histogram           */
/* hist[i * window + d] (d = distance - 1) gets                               */
/*   w_i = (float) sum_{d = 0 .. window-1} (double) wd[d] * (double) hist[.]  */
/* summed in double in ascending d, each product and sum rounded once (no     */
/* fused multiply-add), then rounded once to float.                           */
/* ------------------------------------------------------------------------- */
int oracle_cocount_weights(const int32_t *hist, int64_t n, int32_t window, const float *wd,
                           float *out) {
    if (n < 0 || window < 1 || !wd || (n > 0 && (!hist || !out))) return OR_EINVAL;
    for (int32_t d = 0; d < window; ++d)
        if (!(wd[d] >= 0.0f && wd[d] <= 3.4028234663852886e38f)) return OR_EINVAL;
    for (int64_t i = 0; i < n; ++i) {
        double sum = 0.0;
        for (int32_t d = 0; d < window; ++d) {
            const int32_t h = hist[i * window + d];
            if (h < 0) return OR_ECOUNT;
            const double prod = (double)wd[d] * (double)h;
            sum = sum + prod;
        }
        out[i] = (float)sum;
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Random-walk co-occurrence sampler (Sec. 3.2, Alg. 1).                      */
/*                                                                           */
/* Every seed node s is repeated walks_per_node (gamma) times; walk r of s    */
/* takes walk_steps (k) uniform steps: w_0 = s, and w_t is neighbour          */
/* floor(x * deg / 2^64) of w_{t-1} in CSR order, x = (r1 << 32) | r0 of      */
/* Philox4x32-10 on counter (lo32 s, hi32 s, r, 4 + t) under the seed's key;  */
/* a node without neighbours ends the walk.  The walks of one seed are        */
/* grouped and their co-occurrences combined (Alg. 1, GroupByKey and          */
/* CombineValues):                                                           */
/*   seed_only = 1: the pairs (s, w_t), t = 1 .. window, as in the paper      */
/*                  (the histogram is indexed by the distance t from s);      */
/*   seed_only = 0: every ordered pair (w_a, w_b) of a walk with              */
/*                  1 <= |a - b| <= window (DeepWalk's window), distance      */
/*                  |a - b|.                                                  */
/* Pairs of a node with itself are dropped.  Output: one triple per distinct  */
/* (source, destination) of a seed, seeds in ascending order and, within a   */
/* seed, (source, destination) ascending; cc = number of co-occurrences,      */
/* hist[d - 1] = those at distance d (window entries per triple).             */
/* Returns -4 with *count_out = the number needed if capacity is too small.   */
/* ------------------------------------------------------------------------- */
#define OR_ECAP (-4)

typedef struct {
    int32_t src, dst, dist;
} walk_pair;

static int cmp_walk_pair(const void *a, const void *b) {
    const walk_pair *x = (const walk_pair *)a, *y = (const walk_pair *)b;
    if (x->src != y->src) return x->src < y->src ? -1 : 1;
    if (x->dst != y->dst) return x->dst < y->dst ? -1 : 1;
    if (x->dist != y->dist) return x->dist < y->dist ? -1 : 1;
    return 0;
}

/* One walk; returns its last position (0 .. walk_steps), or -1 on a bad graph. */
static int32_t oracle_walk(const int64_t *off, const int32_t *nbr, int64_t num_nodes,
                           int64_t num_edges, uint64_t seed, int64_t s, int32_t r,
                           int32_t walk_steps, int32_t *w) {
    uint32_t key[2], ctr[4], rr[4];
    seed_key(seed, key);
    w[0] = (int32_t)s;
    for (int32_t t = 1; t <= walk_steps; ++t) {
        const int64_t cur = w[t - 1];
        const int64_t b = off[cur], e = off[cur + 1];
        if (b < 0 || e < b || e > num_edges) return -1;
        const uint64_t deg = (uint64_t)(e - b);
        if (deg == 0) return t - 1;
        ctr[0] = (uint32_t)((uint64_t)s & 0xFFFFFFFFu);
        ctr[1] = (uint32_t)((uint64_t)s >> 32);
        ctr[2] = (uint32_t)r;
        ctr[3] = 4u + (uint32_t)t;
        oracle_philox4x32_10(ctr, key, rr);
        const uint64_t x = ((uint64_t)rr[1] << 32) | (uint64_t)rr[0];
        const uint64_t j = (uint64_t)(((unsigned __int128)x * (unsigned __int128)deg) >> 64);
        const int64_t next = nbr[b + (int64_t)j];
        if (next < 0 || next >= num_nodes) return -1;
        w[t] = (int32_t)next;
    }
    return walk_steps;
}

int oracle_sample_walks(const int64_t *off, const int32_t *nbr, int64_t num_nodes,
                        int64_t num_edges, int32_t walks_per_node, int32_t walk_steps,
                        int32_t window, int32_t seed_only, uint64_t seed, int64_t first_seed,
                        int64_t num_seeds, int32_t *src, int32_t *dst, int32_t *cc,
                        int32_t *hist, int64_t capacity, int64_t *count_out) {
    if (!off || (num_edges > 0 && !nbr) || num_nodes < 1 || num_edges < 0 ||
        walks_per_node < 1 || walk_steps < 1 || window < 1 || window > walk_steps ||
        num_seeds < 0 || first_seed < 0 || first_seed + num_seeds > num_nodes || capacity < 0 ||
        !count_out || (capacity > 0 && (!src || !dst || !cc)))
        return OR_EINVAL;
    int32_t *w = (int32_t *)malloc(sizeof(int32_t) * (size_t)(walk_steps + 1));
    /* pairs of one seed: at most walks * (walk_steps + 1)^2 */
    const int64_t max_pairs =
        (int64_t)walks_per_node * (int64_t)(walk_steps + 1) * (int64_t)(walk_steps + 1);
    walk_pair *pairs = (walk_pair *)malloc(sizeof(walk_pair) * (size_t)max_pairs);
    if (!w || !pairs) {
        free(w); free(pairs);
        return OR_EINVAL;
    }
    int64_t out = 0;
    int rc = OR_OK;
    for (int64_t s = first_seed; s < first_seed + num_seeds && rc == OR_OK; ++s) {
        int64_t np = 0;
        for (int32_t r = 0; r < walks_per_node; ++r) {
            const int32_t last = oracle_walk(off, nbr, num_nodes, num_edges, seed, s, r,
                                             walk_steps, w);
            if (last < 0) {
                rc = OR_ERANGE;
                break;
            }
            for (int32_t a = 0; a <= last; ++a) {
                if (seed_only && a > 0) break;
                for (int32_t b = 0; b <= last; ++b) {
                    const int32_t d = a > b ? a - b : b - a;
                    if (d < 1 || d > window) continue;
                    if (seed_only && b < a) continue;
                    if (w[a] == w[b]) continue;
                    pairs[np].src = w[a];
                    pairs[np].dst = w[b];
                    pairs[np].dist = d;
                    ++np;
                }
            }
        }
        if (rc != OR_OK) break;
        qsort(pairs, (size_t)np, sizeof(walk_pair), cmp_walk_pair);
        for (int64_t i = 0; i < np;) {
            int64_t j = i;
            while (j < np && pairs[j].src == pairs[i].src && pairs[j].dst == pairs[i].dst) ++j;
            if (out < capacity) {
                src[out] = pairs[i].src;
                dst[out] = pairs[i].dst;
                cc[out] = (int32_t)(j - i);
                if (hist) {
                    for (int32_t d = 0; d < window; ++d) hist[out * window + d] = 0;
                    for (int64_t q = i; q < j; ++q) hist[out * window + pairs[q].dist - 1] += 1;
                }
            }
            ++out;
            i = j;
        }
    }
    free(w);
    free(pairs);
    *count_out = out;
    if (rc != OR_OK) return rc;
    return out > capacity ? OR_ECAP : OR_OK;
}

/* ------------------------------------------------------------------------- */
/* Evaluation pairs (Sec. 4's unsupervised metrics: the edge SNR compares    */
/* distances over edges with distances over a random sub-sample of the       */
/* non-edges).  Pair j of the edge sample takes Philox counter               */
/* (lo32 j, hi32 j, 0, 0x80000001): edge index e = floor(x E / 2^64) with     */
/* x = (r1 << 32) | r0 over the E directed edges of the CSR lists, and the   */
/* pair is (the row whose list holds e, nbr[e]).  Pair j of the non-edge     */
/* sample tries a = 0 .. max_tries - 1 with counter (lo32 j, hi32 j, a,      */
/* 0x80000002): u = floor(x0 N / 2^64), v = floor(x1 N / 2^64) with           */
/* x0 = (r1 << 32) | r0 and x1 = (r3 << 32) | r2, and keeps the first try     */
/* with u != v and v not in u's list; with none, the pair is (-1, -1).        */
/* Output: edge pairs at 0 .. n_edge - 1, non-edge pairs after them.          */
/* ------------------------------------------------------------------------- */
static uint64_t mul_hi_u64(uint64_t x, uint64_t n) {
    return (uint64_t)(((unsigned __int128)x * (unsigned __int128)n) >> 64);
}

int oracle_eval_pairs(const int64_t *off, const int32_t *nbr, int64_t num_nodes,
                      int64_t num_edges, uint64_t seed, int64_t n_edge, int64_t n_non,
                      int32_t max_tries, int32_t *u_out, int32_t *v_out) {
    if (!off || num_nodes < 1 || num_edges < 0 || n_edge < 0 || n_non < 0 || max_tries < 1 ||
        (num_edges > 0 && !nbr) || (n_edge + n_non > 0 && (!u_out || !v_out)) ||
        (n_edge > 0 && num_edges == 0) || off[0] != 0 || off[num_nodes] != num_edges)
        return OR_EINVAL;
    uint32_t key[2], ctr[4], r[4];
    seed_key(seed, key);
    for (int64_t j = 0; j < n_edge; ++j) {
        ctr[0] = (uint32_t)((uint64_t)j & 0xFFFFFFFFu);
        ctr[1] = (uint32_t)((uint64_t)j >> 32);
        ctr[2] = 0u;
        ctr[3] = 0x80000001u;
        oracle_philox4x32_10(ctr, key, r);
        const uint64_t x = ((uint64_t)r[1] << 32) | (uint64_t)r[0];
        const int64_t e = (int64_t)mul_hi_u64(x, (uint64_t)num_edges);
        /* the row whose list holds e: the last row with off[row] <= e, by
           bisection over the non-decreasing offsets */
        int64_t lo = 0, hi = num_nodes;  /* off[lo] <= e < off[hi] */
        while (hi - lo > 1) {
            const int64_t mid = lo + (hi - lo) / 2;
            if (off[mid] <= e) lo = mid; else hi = mid;
        }
        const int32_t v = nbr[e];
        if (v < 0 || v >= num_nodes) return OR_ERANGE;
        u_out[j] = (int32_t)lo;
        v_out[j] = v;
    }
    for (int64_t j = 0; j < n_non; ++j) {
        int32_t pu = -1, pv = -1;
        for (int32_t a = 0; a < max_tries; ++a) {
            ctr[0] = (uint32_t)((uint64_t)j & 0xFFFFFFFFu);
            ctr[1] = (uint32_t)((uint64_t)j >> 32);
            ctr[2] = (uint32_t)a;
            ctr[3] = 0x80000002u;
            oracle_philox4x32_10(ctr, key, r);
            const uint64_t x0 = ((uint64_t)r[1] << 32) | (uint64_t)r[0];
            const uint64_t x1 = ((uint64_t)r[3] << 32) | (uint64_t)r[2];
            const int64_t u = (int64_t)mul_hi_u64(x0, (uint64_t)num_nodes);
            const int64_t v = (int64_t)mul_hi_u64(x1, (uint64_t)num_nodes);
            if (u == v) continue;
            int is_edge = 0;
            for (int64_t q = off[u]; q < off[u + 1]; ++q) {
                if (nbr[q] == v) {
                    is_edge = 1;
                    break;
                }
            }
            if (is_edge) continue;
            pu = (int32_t)u;
            pv = (int32_t)v;
            break;
        }
        u_out[n_edge + j] = pu;
        v_out[n_edge + j] = pv;
    }
    return OR_OK;
}

/* ------------------------------------------------------------------------- */
/* bfloat16 tables (the paper's TPUs compute in half precision, Sec. 2.3).    */
/* A bf16 value is a float32 whose 16 low mantissa bits are zero: 1 sign bit, */
/* 8 exponent bits, 7 mantissa bits; stored as its 16 high bits.             */
/* ------------------------------------------------------------------------- */
/* The bf16 nearest to x (ties to the even mantissa), from x itself: no       */
/* intermediate rounding to float.  Overflow gives infinity, NaN a quiet NaN. */
uint16_t oracle_bf16_from_double(double x) {
    if (x != x) return 0x7FC0u;
    const uint16_t sign = signbit(x) ? 0x8000u : 0u;
    const double a = fabs(x);
    if (a == 0.0) return sign;
    int e;
    frexp(a, &e);           /* a in [2^(e-1), 2^e) */
    int E = e - 1;
    if (E < -126) E = -126; /* subnormals share the smallest quantum */
    const double q = ldexp(1.0, E - 7);
    const double r = a / q; /* exact: q is a power of two */
    double n = floor(r);
    const double frac = r - n;
    if (frac > 0.5 || (frac == 0.5 && fmod(n, 2.0) != 0.0)) n += 1.0;
    const double v = n * q;
    if (v >= ldexp(1.0, 128)) return (uint16_t)(sign | 0x7F80u);
    const float f = (float)v; /* exact: v is a bf16 value */
    uint32_t bits;
    memcpy(&bits, &f, 4);
    return (uint16_t)(sign | (uint16_t)(bits >> 16));
}

double oracle_bf16_to_double(uint16_t h) {
    const uint32_t bits = (uint32_t)h << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

/* Initial rows of bf16 tables: the float initial values rounded to bf16. */
int oracle_init_rows_bf16(uint64_t seed, int32_t table, const int64_t *rows, int64_t nrows,
                          int32_t dim, float half_width, uint16_t *out) {
    if (nrows < 0 || dim <= 0 || (nrows > 0 && (!rows || !out))) return OR_EINVAL;
    float *tmp = (float *)malloc(sizeof(float) * (size_t)dim);
    if (!tmp) return OR_EINVAL;
    for (int64_t r = 0; r < nrows; ++r) {
        int rc = oracle_init_rows(seed, table, rows + r, 1, dim, half_width, tmp);
        if (rc) { free(tmp); return rc; }
        for (int32_t d = 0; d < dim; ++d)
            out[r * dim + d] = oracle_bf16_from_double((double)tmp[d]);
    }
    free(tmp);
    return OR_OK;
}

/* One step on bf16 tables: widened to double, the same gradient as the float
   step, and each touched element rewritten once as
   bf16_nearest((double)row - (double)lr * grad).  cc or wf as in the float
   steps (exactly one given). */
int oracle_sgns_step_bf16(uint16_t *S, uint16_t *T, int64_t ns, int64_t nt, int32_t dim,
                          int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                          const int32_t *cc, const float *wf, const int32_t *neg, float lr,
                          double *loss_out) {
    if (!S || !T || dim <= 0 || n < 0 || num_neg < 1 || !loss_out) return OR_EINVAL;
    if (n > 0 && (!src || !dst || (!cc && !wf) || !neg)) return OR_EINVAL;
    int rc = check_batch(ns, nt, n, num_neg, src, dst, cc, wf, neg);
    if (rc) return rc;
    size_t s_elems = (size_t)ns * (size_t)dim, t_elems = (size_t)nt * (size_t)dim;
    double *Sd = (double *)malloc(s_elems * sizeof(double));
    double *Td = (double *)malloc(t_elems * sizeof(double));
    double *gS = (double *)malloc(s_elems * sizeof(double));
    double *gT = (double *)malloc(t_elems * sizeof(double));
    unsigned char *touched_S = (unsigned char *)calloc((size_t)ns, 1);
    unsigned char *touched_T = (unsigned char *)calloc((size_t)nt, 1);
    if (!Sd || !Td || !gS || !gT || !touched_S || !touched_T) {
        free(Sd); free(Td); free(gS); free(gT); free(touched_S); free(touched_T);
        return OR_EINVAL;
    }
    for (size_t e = 0; e < s_elems; ++e) Sd[e] = oracle_bf16_to_double(S[e]);
    for (size_t e = 0; e < t_elems; ++e) Td[e] = oracle_bf16_to_double(T[e]);
    double loss = 0.0;
    rc = sgns_grad_d(Sd, Td, ns, nt, dim, n, num_neg, src, dst, cc, wf, neg, gS, gT, &loss);
    if (rc == OR_OK) {
        for (int64_t i = 0; i < n; ++i) {
            touched_S[src[i]] = 1;
            touched_T[dst[i]] = 1;
            for (int32_t k = 0; k < num_neg; ++k) touched_T[neg[i * num_neg + k]] = 1;
        }
        const double lr_d = (double)lr;
        for (int64_t r = 0; r < ns; ++r)
            if (touched_S[r])
                for (int32_t d = 0; d < dim; ++d)
                    S[r * dim + d] =
                        oracle_bf16_from_double(Sd[r * dim + d] - lr_d * gS[r * dim + d]);
        for (int64_t r = 0; r < nt; ++r)
            if (touched_T[r])
                for (int32_t d = 0; d < dim; ++d)
                    T[r * dim + d] =
                        oracle_bf16_from_double(Td[r * dim + d] - lr_d * gT[r * dim + d]);
        *loss_out = loss;
    }
    free(Sd); free(Td); free(gS); free(gT); free(touched_S); free(touched_T);
    return rc;
}
