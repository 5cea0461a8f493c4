/*
 * Sanitizer driver for the CPU oracle (test infrastructure): calls every
 * exported oracle routine on small inputs -- valid ones, the empty batch,
 * repeated rows, weights, bf16 tables, walks, evaluation pairs -- and the
 * argument errors, so that AddressSanitizer and UndefinedBehaviorSanitizer
 * see each code path.  Built and run by tests/test_sanitize.py; exits 0 when
 * every call returns what it should (the sanitizers abort on a finding).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void oracle_philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]);
int oracle_init_rows(uint64_t seed, int32_t table, const int64_t *rows, int64_t nrows,
                     int32_t dim, float half_width, float *out);
int oracle_build_alias(const double *weights, int64_t n, uint32_t *thr, int32_t *alias);
int64_t oracle_sample_negative(uint64_t seed, uint64_t p, int32_t k, int64_t num_nodes,
                               const uint32_t *thr, const int32_t *alias);
int oracle_sample_negatives(uint64_t seed, uint64_t first_pos, int64_t n, int32_t num_neg,
                            int64_t num_nodes, const uint32_t *thr, const int32_t *alias,
                            int32_t *neg_out);
int oracle_sgns_grad_d(const double *S, const double *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const int32_t *cc, const int32_t *neg, double *grad_S, double *grad_T,
                       double *loss_out);
int oracle_sgns_loss_d(const double *S, const double *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const int32_t *cc, const int32_t *neg, double *loss_out);
int oracle_sgns_step(float *S, float *T, int64_t ns, int64_t nt, int32_t dim, int64_t n,
                     int32_t num_neg, const int32_t *src, const int32_t *dst, const int32_t *cc,
                     const int32_t *neg, float lr, double *loss_out);
int oracle_sgns_step_w(float *S, float *T, int64_t ns, int64_t nt, int32_t dim, int64_t n,
                       int32_t num_neg, const int32_t *src, const int32_t *dst, const float *w,
                       const int32_t *neg, float lr, double *loss_out);
int oracle_sgns_loss(const float *S, const float *T, int64_t ns, int64_t nt, int32_t dim,
                     int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                     const int32_t *cc, const int32_t *neg, double *loss_out);
int oracle_sgns_loss_w(const float *S, const float *T, int64_t ns, int64_t nt, int32_t dim,
                       int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                       const float *w, const int32_t *neg, double *loss_out);
int oracle_cocount_weights(const int32_t *hist, int64_t n, int32_t window, const float *wd,
                           float *out);
int oracle_sample_walks(const int64_t *off, const int32_t *nbr, int64_t num_nodes,
                        int64_t num_edges, int32_t walks_per_node, int32_t walk_steps,
                        int32_t window, int32_t seed_only, uint64_t seed, int64_t first_seed,
                        int64_t num_seeds, int32_t *src, int32_t *dst, int32_t *cc,
                        int32_t *hist, int64_t capacity, int64_t *count_out);
int oracle_eval_pairs(const int64_t *off, const int32_t *nbr, int64_t num_nodes,
                      int64_t num_edges, uint64_t seed, int64_t n_edge, int64_t n_non,
                      int32_t max_tries, int32_t *u_out, int32_t *v_out);
uint16_t oracle_bf16_from_double(double x);
double oracle_bf16_to_double(uint16_t h);
int oracle_init_rows_bf16(uint64_t seed, int32_t table, const int64_t *rows, int64_t nrows,
                          int32_t dim, float half_width, uint16_t *out);
int oracle_sgns_step_bf16(uint16_t *S, uint16_t *T, int64_t ns, int64_t nt, int32_t dim,
                          int64_t n, int32_t num_neg, const int32_t *src, const int32_t *dst,
                          const int32_t *cc, const float *wf, const int32_t *neg, float lr,
                          double *loss_out);

static int failures = 0;
#define EXPECT(cond)                                                         \
    do {                                                                     \
        if (!(cond)) {                                                       \
            fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__,     \
                    __LINE__, #cond);                                        \
            ++failures;                                                      \
        }                                                                    \
    } while (0)

enum { NN = 37, DIM = 20, NB = 50, KN = 3 };

int main(void) {
    /* Philox */
    uint32_t ctr[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    oracle_philox4x32_10(ctr, key, out);

    /* tables (every row), float and double copies */
    int64_t ids[NN];
    for (int64_t j = 0; j < NN; ++j) ids[j] = j;
    float *S = malloc(sizeof(float) * NN * DIM), *T = malloc(sizeof(float) * NN * DIM);
    EXPECT(oracle_init_rows(11, 0, ids, NN, DIM, 0.5f, S) == 0);
    EXPECT(oracle_init_rows(11, 1, ids, NN, DIM, 0.5f, T) == 0);
    EXPECT(oracle_init_rows(11, 0, ids, -1, DIM, 0.5f, S) != 0);
    double *Sd = malloc(sizeof(double) * NN * DIM), *Td = malloc(sizeof(double) * NN * DIM);
    for (int j = 0; j < NN * DIM; ++j) {
        Sd[j] = S[j];
        Td[j] = T[j];
    }

    /* alias table over skewed weights (one zero), and its errors */
    double w[NN];
    for (int j = 0; j < NN; ++j) w[j] = (j % 5 == 0) ? 7.0 : (j == 3 ? 0.0 : 1.0 + j);
    uint32_t thr[NN];
    int32_t alias[NN];
    EXPECT(oracle_build_alias(w, NN, thr, alias) == 0);
    for (int j = 0; j < NN; ++j) EXPECT(alias[j] >= 0 && alias[j] < NN);
    EXPECT(oracle_build_alias(w, 0, thr, alias) != 0);
    w[1] = -1.0;
    EXPECT(oracle_build_alias(w, NN, thr, alias) != 0);
    w[1] = 2.0;

    /* a batch with repeated rows (src and dst drawn from few ids) */
    int32_t src[NB], dst[NB], cc[NB], neg[NB * KN], negw[NB * KN];
    float wf[NB];
    for (int i = 0; i < NB; ++i) {
        src[i] = (i * 7) % 11;
        dst[i] = (i * 5 + 3) % NN;
        cc[i] = 1 + i % 4;
        wf[i] = 0.25f * (float)(1 + i % 3);
    }
    EXPECT(oracle_sample_negatives(3, 100, NB, KN, NN, NULL, NULL, neg) == 0);
    EXPECT(oracle_sample_negatives(3, 100, NB, KN, NN, thr, alias, negw) == 0);
    for (int j = 0; j < NB * KN; ++j) EXPECT(neg[j] >= 0 && neg[j] < NN && negw[j] >= 0 && negw[j] < NN);
    EXPECT(oracle_sample_negative(3, 1ull << 40, 2, NN, thr, alias) < NN);
    EXPECT(oracle_sample_negatives(3, 100, NB, 0, NN, NULL, NULL, neg) != 0);

    double loss = 0.0;
    double *gS = calloc(NN * DIM, sizeof(double)), *gT = calloc(NN * DIM, sizeof(double));
    EXPECT(oracle_sgns_grad_d(Sd, Td, NN, NN, DIM, NB, KN, src, dst, cc, neg, gS, gT, &loss) == 0);
    EXPECT(oracle_sgns_loss_d(Sd, Td, NN, NN, DIM, NB, KN, src, dst, cc, neg, &loss) == 0);
    EXPECT(oracle_sgns_loss(S, T, NN, NN, DIM, NB, KN, src, dst, cc, neg, &loss) == 0);
    EXPECT(oracle_sgns_loss_w(S, T, NN, NN, DIM, NB, KN, src, dst, wf, neg, &loss) == 0);
    EXPECT(oracle_sgns_step(S, T, NN, NN, DIM, NB, KN, src, dst, cc, neg, 0.025f, &loss) == 0);
    EXPECT(oracle_sgns_step_w(S, T, NN, NN, DIM, NB, KN, src, dst, wf, negw, 0.025f, &loss) == 0);
    EXPECT(oracle_sgns_step(S, T, NN, NN, DIM, 0, KN, src, dst, cc, neg, 0.025f, &loss) == 0);
    /* errors: an id out of range, a negative co_count */
    src[4] = NN;
    EXPECT(oracle_sgns_step(S, T, NN, NN, DIM, NB, KN, src, dst, cc, neg, 0.025f, &loss) != 0);
    src[4] = 0;
    cc[7] = -1;
    EXPECT(oracle_sgns_loss(S, T, NN, NN, DIM, NB, KN, src, dst, cc, neg, &loss) != 0);
    cc[7] = 1;

    /* co_count weights from distance histograms */
    enum { WIN = 4 };
    int32_t hist[NB * WIN];
    float wd[WIN] = {1.0f, 0.5f, 0.25f, 0.125f}, wout[NB];
    for (int j = 0; j < NB * WIN; ++j) hist[j] = j % 3;
    EXPECT(oracle_cocount_weights(hist, NB, WIN, wd, wout) == 0);
    hist[5] = -2;
    EXPECT(oracle_cocount_weights(hist, NB, WIN, wd, wout) != 0);

    /* bf16 tables */
    uint16_t *Sb = malloc(sizeof(uint16_t) * NN * DIM), *Tb = malloc(sizeof(uint16_t) * NN * DIM);
    EXPECT(oracle_init_rows_bf16(11, 0, ids, NN, DIM, 0.5f, Sb) == 0);
    EXPECT(oracle_init_rows_bf16(11, 1, ids, NN, DIM, 0.5f, Tb) == 0);
    EXPECT(oracle_sgns_step_bf16(Sb, Tb, NN, NN, DIM, NB, KN, src, dst, cc, NULL, neg, 0.025f, &loss) == 0);
    EXPECT(oracle_sgns_step_bf16(Sb, Tb, NN, NN, DIM, NB, KN, src, dst, NULL, wf, neg, 0.025f, &loss) == 0);
    EXPECT(oracle_bf16_to_double(oracle_bf16_from_double(1.0)) == 1.0);
    (void)oracle_bf16_from_double(1e39);
    (void)oracle_bf16_from_double(-3e-40);

    /* a ring of 12 nodes with chords; one node without edges */
    enum { GN = 13 };
    int64_t off[GN + 1];
    int32_t nbr[64];
    int64_t e = 0;
    for (int u = 0; u < GN; ++u) {
        off[u] = e;
        if (u == GN - 1) continue;
        nbr[e++] = (u + 1) % (GN - 1);
        nbr[e++] = (u + GN - 2) % (GN - 1);
        if (u % 3 == 0) nbr[e++] = (u + 5) % (GN - 1);
    }
    off[GN] = e;
    enum { CAP = 4096 };
    int32_t *ws = malloc(sizeof(int32_t) * CAP), *wd2 = malloc(sizeof(int32_t) * CAP);
    int32_t *wc = malloc(sizeof(int32_t) * CAP), *wh = malloc(sizeof(int32_t) * CAP * 3);
    int64_t count = 0;
    EXPECT(oracle_sample_walks(off, nbr, GN, e, 2, 6, 3, 0, 9, 0, GN, ws, wd2, wc, wh, CAP, &count) == 0);
    EXPECT(count > 0 && count <= CAP);
    EXPECT(oracle_sample_walks(off, nbr, GN, e, 2, 6, 3, 1, 9, 2, 5, ws, wd2, wc, NULL, CAP, &count) == 0);
    EXPECT(oracle_sample_walks(off, nbr, GN, e, 2, 6, 3, 0, 9, 0, GN, ws, wd2, wc, wh, 4, &count) != 0);
    EXPECT(oracle_sample_walks(off, nbr, GN, e, 2, 6, 9, 0, 9, 0, GN, ws, wd2, wc, wh, CAP, &count) != 0);

    int32_t pu[40], pv[40];
    EXPECT(oracle_eval_pairs(off, nbr, GN, e, 4, 20, 20, 64, pu, pv) == 0);
    for (int j = 0; j < 40; ++j) EXPECT(pu[j] >= -1 && pu[j] < GN && pv[j] >= -1 && pv[j] < GN);
    EXPECT(oracle_eval_pairs(off, nbr, GN, e, 4, 20, 20, 0, pu, pv) != 0);

    free(S); free(T); free(Sd); free(Td); free(gS); free(gT); free(Sb); free(Tb);
    free(ws); free(wd2); free(wc); free(wh);
    if (failures) {
        fprintf(stderr, "%d expectation(s) failed\n", failures);
        return 1;
    }
    printf("oracle sanitizer drive: ok\n");
    return 0;
}
