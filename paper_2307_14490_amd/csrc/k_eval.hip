// Unsupervised evaluation of an embedding table (HUGE Sec. 4): the rows are
// L2-normalised and compared by Euclidean distance;
//   - edge SNR: mean distance over a random sample of non-edges divided by the
//     mean over a sample of edges, with the distribution of both (percentiles);
//   - sampled edge recall: for a few query nodes u, the k rows nearest to u
//     form S, and recall@k(u) = |N(u) & S| / k.
// Kernels:
//   k_eval_pairs    edge and non-edge pairs from counter-based Philox draws
//   k_eval_dist     distances of normalised rows, G lanes per pair
//   k_eval_sums     per-block double sums and counts of the valid distances;
//   k_eval_final    their fixed-order totals, the means and the SNR;
//   k_eval_quantile percentiles of the sorted distances (sorted by the radix
//                   kernels of k_sort.hip on the float bit patterns);
//   k_knn_queries   the normalised query rows;
//   k_knn_tiles_h   distances of every row to every query (32 queries x 32 rows
//                   per tile) for dim <= 128: rows and queries split into two
//                   fp16 parts on the fp16 matrix cores; per-wave top-k lists;
//   k_knn_tiles     the same for wider rows: fp32 matrix cores, queries in LDS;
//   k_knn_merge     the k nearest of each query over all lists (bitonic sort);
//   k_eval_recall   recall@k from the nearest rows and the sorted CSR lists.
#include "common.hpp"
#include "device.hpp"
#include "dispatch.hpp"

namespace huge {

__device__ __forceinline__ void eval_fail(int32_t* status, int32_t code) {
    atomicCAS(status, 0, code);
}

// The row whose list holds edge e: the last row r with off[r] <= e, by
// bisection over the offsets (off[0] = 0 <= e < off[N] = E).
__device__ __forceinline__ int64_t edge_row(const int64_t* __restrict__ off, int64_t N,
                                            int64_t e) {
    int64_t lo = 0, hi = N;
    while (hi - lo > 1) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (off[mid] <= e)
            lo = mid;
        else
            hi = mid;
    }
    return lo;
}

// Whether v is in the ascending list nbr[b, e).
__device__ __forceinline__ bool in_sorted_list(const int32_t* __restrict__ nbr, int64_t b,
                                               int64_t e, int32_t v) {
    while (b < e) {
        const int64_t mid = b + (e - b) / 2;
        const int32_t x = nbr[mid];
        if (x == v) return true;
        if (x < v)
            b = mid + 1;
        else
            e = mid;
    }
    return false;
}

// ---------------------------------------------------------------------------
// Pairs.  Edge pair j: Philox counter (lo32 j, hi32 j, 0, kEdgeWord), edge
// index floor(x E / 2^64) with x = (r1 << 32) | r0, the pair (its row, its
// neighbour).  Non-edge pair j: tries a = 0 .. max_tries - 1 with counter
// (lo32 j, hi32 j, a, kNonEdgeWord), u = floor(x0 N / 2^64), v =
// floor(x1 N / 2^64) (x0 = (r1 << 32) | r0, x1 = (r3 << 32) | r2); the first
// try with u != v and v not in u's list, else (-1, -1).
// ---------------------------------------------------------------------------
constexpr uint32_t kEdgeWord = 0x80000001u;
constexpr uint32_t kNonEdgeWord = 0x80000002u;

__global__ __launch_bounds__(kBlock) void k_eval_pairs(
    const int64_t* __restrict__ off, const int32_t* __restrict__ nbr, int64_t N, int64_t E,
    uint64_t seed, int64_t n_edge, int64_t n_non, int32_t max_tries, int32_t* __restrict__ u_out,
    int32_t* __restrict__ v_out, int32_t* __restrict__ status) {
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (j >= n_edge + n_non) return;
    const uint32_t klo = (uint32_t)seed, khi = (uint32_t)(seed >> 32);
    int32_t pu = -1, pv = -1;
    if (j < n_edge) {
        const uint4 r = philox4x32_10(make_uint4((uint32_t)j, (uint32_t)((uint64_t)j >> 32), 0u,
                                                 kEdgeWord), klo, khi);
        const uint64_t x = ((uint64_t)r.y << 32) | r.x;
        const int64_t e = (int64_t)__umul64hi(x, (uint64_t)E);
        const int64_t row = edge_row(off, N, e);
        const int32_t v = nbr[e];
        if (off[row] <= e && e < off[row + 1] && v >= 0 && (int64_t)v < N) {
            pu = (int32_t)row;
            pv = v;
        } else {
            eval_fail(status, -2);
        }
    } else {
        const int64_t jj = j - n_edge;
        for (int32_t a = 0; a < max_tries; ++a) {
            const uint4 r = philox4x32_10(
                make_uint4((uint32_t)jj, (uint32_t)((uint64_t)jj >> 32), (uint32_t)a,
                           kNonEdgeWord), klo, khi);
            const int64_t u = (int64_t)__umul64hi(((uint64_t)r.y << 32) | r.x, (uint64_t)N);
            const int64_t v = (int64_t)__umul64hi(((uint64_t)r.w << 32) | r.z, (uint64_t)N);
            if (u == v) continue;
            const int64_t b = off[u], e = off[u + 1];
            if (b < 0 || e < b || e > E) {
                eval_fail(status, -2);
                break;
            }
            if (in_sorted_list(nbr, b, e, (int32_t)v)) continue;
            pu = (int32_t)u;
            pv = (int32_t)v;
            break;
        }
    }
    u_out[j] = pu;
    v_out[j] = pv;
}

hipError_t launch_eval_pairs(const int64_t* off, const int32_t* nbr, int64_t N, int64_t E,
                             uint64_t seed, int64_t n_edge, int64_t n_non, int32_t max_tries,
                             int32_t* u, int32_t* v, int32_t* status, hipStream_t s) {
    const int64_t n = n_edge + n_non;
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_eval_pairs, dim3((unsigned)((n + kBlock - 1) / kBlock)), dim3(kBlock),
                       0, s, off, nbr, N, E, seed, n_edge, n_non, max_tries, u, v, status);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Distances: |x_u / |x_u| - x_v / |x_v||, G lanes per pair and C float4 per
// lane (a zero row stays zero); NaN for a pair with a negative id.
// ---------------------------------------------------------------------------
template <int G, int C>
__global__ __launch_bounds__(kBlock) void k_eval_dist(const float* __restrict__ T, int64_t N,
                                                      int32_t D, const int32_t* __restrict__ u,
                                                      const int32_t* __restrict__ v, int64_t n,
                                                      float* __restrict__ out,
                                                      int32_t* __restrict__ status) {
    const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int64_t p = t / G;  // groups are aligned in the wave and exit together
    const int g = (int)(t % G);
    if (p >= n) return;
    const int32_t a = u[p], b = v[p];
    if (a < 0 || b < 0) {
        if (g == 0) out[p] = __builtin_nanf("");
        return;
    }
    if ((int64_t)a >= N || (int64_t)b >= N) {
        if (g == 0) {
            out[p] = __builtin_nanf("");
            eval_fail(status, -2);
        }
        return;
    }
    const int q4 = D / 4;
    const float4* xa = reinterpret_cast<const float4*>(T + (int64_t)a * D);
    const float4* xb = reinterpret_cast<const float4*>(T + (int64_t)b * D);
    float4 ra[C], rb[C];
    float na = 0.f, nb = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int idx = g + G * c;
        ra[c] = idx < q4 ? xa[idx] : make_float4(0.f, 0.f, 0.f, 0.f);
        rb[c] = idx < q4 ? xb[idx] : make_float4(0.f, 0.f, 0.f, 0.f);
        na += ra[c].x * ra[c].x + ra[c].y * ra[c].y + ra[c].z * ra[c].z + ra[c].w * ra[c].w;
        nb += rb[c].x * rb[c].x + rb[c].y * rb[c].y + rb[c].z * rb[c].z + rb[c].w * rb[c].w;
    }
    na = group_sum<G>(na);
    nb = group_sum<G>(nb);
    const float ia = na > 0.f ? 1.0f / sqrtf(na) : 0.f;
    const float ib = nb > 0.f ? 1.0f / sqrtf(nb) : 0.f;
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const float dx = ra[c].x * ia - rb[c].x * ib, dy = ra[c].y * ia - rb[c].y * ib;
        const float dz = ra[c].z * ia - rb[c].z * ib, dw = ra[c].w * ia - rb[c].w * ib;
        s += dx * dx + dy * dy + dz * dz + dw * dw;
    }
    s = group_sum<G>(s);
    if (g == 0) out[p] = sqrtf(s);
}

hipError_t launch_eval_dist(const float* T, int64_t N, int32_t D, const int32_t* u,
                            const int32_t* v, int64_t n, float* out, int32_t* status,
                            hipStream_t s) {
    if (n == 0) return hipSuccess;
    const RowShape rs = row_shape(D);
    const int64_t threads = n * rs.G;
    const dim3 grid((unsigned)((threads + kBlock - 1) / kBlock));
    HUGE_ROW_DISPATCH(rs, hipLaunchKernelGGL((k_eval_dist<G_, C_>), grid, dim3(kBlock), 0, s, T,
                                             N, D, u, v, n, out, status));
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Summary of n_edge edge distances followed by n_non non-edge distances:
// counts and sums of the non-NaN values per block (fixed tree order), then
// out[0..4] = count_edge, count_non, mean_edge, mean_non, mean_non / mean_edge.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_eval_sums(const float* __restrict__ d, int64_t n_edge,
                                                      int64_t n, double* __restrict__ part) {
    __shared__ double s_v[4][kBlock];
    double se = 0.0, sn = 0.0, ce = 0.0, cn = 0.0;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kBlock) {
        const float x = d[i];
        if (x != x) continue;
        if (i < n_edge) {
            se += x;
            ce += 1.0;
        } else {
            sn += x;
            cn += 1.0;
        }
    }
    s_v[0][threadIdx.x] = se;
    s_v[1][threadIdx.x] = sn;
    s_v[2][threadIdx.x] = ce;
    s_v[3][threadIdx.x] = cn;
    __syncthreads();
    for (int w = kBlock / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w)
            for (int c = 0; c < 4; ++c) s_v[c][threadIdx.x] += s_v[c][threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x < 4) part[blockIdx.x * 4 + threadIdx.x] = s_v[threadIdx.x][0];
}

__global__ void k_eval_final(const double* __restrict__ part, int blocks, double* __restrict__ out) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    double t[4] = {0.0, 0.0, 0.0, 0.0};
    for (int b = 0; b < blocks; ++b)
        for (int c = 0; c < 4; ++c) t[c] += part[b * 4 + c];
    const double nan = __builtin_nan("");
    const double me = t[2] > 0.0 ? t[0] / t[2] : nan;
    const double mn = t[3] > 0.0 ? t[1] / t[3] : nan;
    out[0] = t[2];
    out[1] = t[3];
    out[2] = me;
    out[3] = mn;
    out[4] = (t[2] > 0.0 && t[3] > 0.0) ? mn / me : nan;
}

// Percentile q of the `count` smallest values of the ascending keys (the
// valid distances; NaN bit patterns sort after them): position
// h = (count - 1) q / 100, linear between the order statistics around h.
struct Quantiles {
    double q[kEvalMaxQuantiles];
};

__global__ void k_eval_quantile(const uint32_t* __restrict__ sorted, const double* __restrict__ cnt,
                                Quantiles Q, int nq, double* __restrict__ out) {
    const int i = threadIdx.x;
    if (i >= nq) return;
    const int64_t count = (int64_t)*cnt;
    if (count <= 0) {
        out[i] = __builtin_nan("");
        return;
    }
    const double h = (double)(count - 1) * (Q.q[i] / 100.0);
    int64_t lo = (int64_t)floor(h);
    if (lo < 0) lo = 0;
    if (lo > count - 1) lo = count - 1;
    const int64_t hi = lo + 1 < count ? lo + 1 : count - 1;
    const double a = (double)__uint_as_float(sorted[lo]);
    const double b = (double)__uint_as_float(sorted[hi]);
    out[i] = a + (h - (double)lo) * (b - a);
}

hipError_t launch_eval_sums(const float* d, int64_t n_edge, int64_t n, double* part, double* out,
                            hipStream_t s) {
    hipLaunchKernelGGL(k_eval_sums, dim3(kEvalSumBlocks), dim3(kBlock), 0, s, d, n_edge, n, part);
    hipLaunchKernelGGL(k_eval_final, dim3(1), dim3(64), 0, s, part, kEvalSumBlocks, out);
    return hipGetLastError();
}

hipError_t launch_eval_quantiles(const uint32_t* sorted, const double* cnt, const double* q,
                                 int nq, double* out, hipStream_t s) {
    if (nq <= 0) return hipSuccess;
    if (nq > kEvalMaxQuantiles) return hipErrorInvalidValue;
    Quantiles Q;
    for (int i = 0; i < nq; ++i) Q.q[i] = q[i];
    hipLaunchKernelGGL(k_eval_quantile, dim3(1), dim3(kEvalMaxQuantiles), 0, s, sorted, cnt, Q,
                       nq, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Nearest rows of up to kKnnPass queries per pass over the table.
// ---------------------------------------------------------------------------
// Normalised query rows qn[j * D ..] (zero for a zero row or a padding slot)
// and qn2[j] = |qn_j|^2 in {0, 1}; with the threshold scans, their state: no
// candidates, the bound +inf (-inf for a padding slot: nothing passes it) and
// the fallback gate closed.
__global__ __launch_bounds__(kBlock) void k_knn_queries(const float* __restrict__ T, int64_t N,
                                                        int32_t D, const int32_t* __restrict__ q,
                                                        int32_t nq, int32_t nqp,
                                                        float* __restrict__ qn,
                                                        float* __restrict__ qn2,
                                                        int32_t* __restrict__ qid,
                                                        float* __restrict__ tau,
                                                        uint32_t* __restrict__ cnt,
                                                        int32_t* __restrict__ gate,
                                                        int32_t* __restrict__ status) {
    __shared__ float s_red[kBlock];
    const int j = blockIdx.x;
    if (j >= nqp) return;
    int32_t id = j < nq ? q[j] : -1;
    if (id >= 0 && (int64_t)id >= N) {
        if (threadIdx.x == 0) eval_fail(status, -2);
        id = -1;
    }
    if (j < nq && id < 0 && q[j] < 0 && threadIdx.x == 0) eval_fail(status, -2);
    float part = 0.f;
    for (int c = threadIdx.x; c < D; c += kBlock) {
        const float x = id >= 0 ? T[(int64_t)id * D + c] : 0.f;
        part += x * x;
    }
    s_red[threadIdx.x] = part;
    __syncthreads();
    for (int w = kBlock / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s_red[threadIdx.x] += s_red[threadIdx.x + w];
        __syncthreads();
    }
    const float n2 = s_red[0];
    const float inv = n2 > 0.f ? 1.0f / sqrtf(n2) : 0.f;
    for (int c = threadIdx.x; c < D; c += kBlock)
        qn[(int64_t)j * D + c] = id >= 0 ? T[(int64_t)id * D + c] * inv : 0.f;
    if (threadIdx.x == 0) {
        qn2[j] = n2 > 0.f ? 1.f : 0.f;
        qid[j] = id;
        if (cnt) {
            cnt[j] = 0u;
            tau[j] = id >= 0 ? __builtin_inff() : -__builtin_inff();
        }
        if (gate && j == 0) *gate = 0;
    }
}

typedef float knn_acc16 __attribute__((ext_vector_type(16)));

// One workgroup of kKnnWaves waves; wave w serves query block w % QB (32
// queries) over tiles t = S, S + NS, ... of 32 rows, S = its list slot.  Per
// tile: the 32 x 32 dot products of the normalised queries with the raw rows
// by v_mfma_f32_32x32x2f32 (the K dimension runs over the dimensions in
// chunks of 128: lane (x, h) supplies row x's dimensions c*128 + h*64 + s and
// query x's same dimension at step s), the rows' norms from the same
// registers, then d^2 = |q|^2 + [row != 0] - 2 dot / |row| and the key
// (bits of d^2) << 32 | row.  Keys below the query's current k-th best are
// staged per query (at most 32 per tile) and inserted by the query's own lane
// into its sorted list of k.  Lists go to partial[(S * nqp + q) * k + t].
struct KnnArgs {
    const float* T;
    int64_t N;
    int32_t D;
    int32_t k;
    int32_t nqp;   // queries in this pass, padded to 32 * QB
    int32_t QB;    // query blocks: 1, 2 or 4
    int32_t stride;  // LDS floats per query row (D + 4)
    int64_t tiles;
    const float* qn;
    const float* qn2;
    const int32_t* qid;
    uint64_t* partial;
    const int32_t* gate;  // null: always run; else run only where *gate != 0
};

constexpr uint64_t kNoKey = ~0ull;

__global__ __launch_bounds__(kKnnWaves * 64) void k_knn_tiles(KnnArgs A) {
    __shared__ __align__(16) float s_q[kKnnQueryFloats];
    __shared__ uint64_t s_list[kKnnWaves][32][kKnnMaxK];
    __shared__ uint64_t s_stage[kKnnWaves][32][32];
    __shared__ uint64_t s_thr[kKnnWaves][32];
    __shared__ uint32_t s_cnt[kKnnWaves][32];
    __shared__ uint32_t s_len[kKnnWaves][32];
    __shared__ float s_qn2[kKnnPass];
    __shared__ int32_t s_qid[kKnnPass];

    if (A.gate && *A.gate == 0) return;  // the threshold scans answered every query
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int x = lane & 31, h = lane >> 5;
    const int D = A.D, k = A.k, stride = A.stride;
    for (int i = tid; i < kKnnQueryFloats; i += kKnnWaves * 64) s_q[i] = 0.f;
    __syncthreads();
    for (int64_t i = tid; i < (int64_t)A.nqp * D; i += kKnnWaves * 64)
        s_q[(i / D) * stride + (i % D)] = A.qn[i];
    for (int i = tid; i < A.nqp; i += kKnnWaves * 64) {
        s_qn2[i] = A.qn2[i];
        s_qid[i] = A.qid[i];
    }
    if (lane < 32) {
        s_thr[w][lane] = kNoKey;
        s_cnt[w][lane] = 0u;
        s_len[w][lane] = 0u;
    }
    __syncthreads();

    const int qb = w % A.QB;
    const int wpb = kKnnWaves / A.QB;  // waves per query block
    const int64_t S = (int64_t)blockIdx.x * wpb + w / A.QB;
    const int64_t NS = (int64_t)gridDim.x * wpb;
    const int nch = (D + kKnnDimChunk - 1) / kKnnDimChunk;
    const float* qrow = s_q + (qb * 32 + x) * stride;

    // one dimension chunk (dim <= 128): the next tile's rows are loaded
    // while the current tile's products run
    constexpr int kQ4 = kKnnDimChunk / 8;  // float4 of a lane's half row
    const int d0h = h * (kKnnDimChunk / 2);
    auto load_rows = [&](int64_t tt, int c, float4* bv) {
        const int64_t rr = tt * 32 + x;
        const int d0 = c * kKnnDimChunk + d0h;
        const float4* src = reinterpret_cast<const float4*>(A.T + rr * (int64_t)D + d0);
        const bool ok = tt < A.tiles && rr < A.N;
#pragma unroll
        for (int m = 0; m < kQ4; ++m)
            bv[m] = (ok && d0 + 4 * m < D) ? src[m] : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    float4 nxt[kQ4];
    if (nch == 1) load_rows(S, 0, nxt);
    for (int64_t t = S; t < A.tiles; t += NS) {
        const int64_t row = t * 32 + x;
        const bool row_ok = row < A.N;
        // two independent accumulation chains (even and odd float4 of the
        // lane's half row), added at the end
        knn_acc16 acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                         0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        knn_acc16 acc1 = acc;
        float nr = 0.f;
        for (int c = 0; c < nch; ++c) {
            const int d0 = c * kKnnDimChunk + d0h;
            float4 bv[kQ4];
            if (nch == 1) {
#pragma unroll
                for (int m = 0; m < kQ4; ++m) bv[m] = nxt[m];
                load_rows(t + NS, 0, nxt);
            } else {
                load_rows(t, c, bv);
            }
#pragma unroll
            for (int m = 0; m < kQ4; ++m) {
                nr += bv[m].x * bv[m].x + bv[m].y * bv[m].y + bv[m].z * bv[m].z +
                      bv[m].w * bv[m].w;
                const int dd = d0 + 4 * m;
                float4 av = make_float4(0.f, 0.f, 0.f, 0.f);
                if (dd < D) av = *reinterpret_cast<const float4*>(qrow + dd);
                if (m % 2 == 0) {
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.x, bv[m].x, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.y, bv[m].y, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.z, bv[m].z, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.w, bv[m].w, acc, 0, 0, 0);
                } else {
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av.x, bv[m].x, acc1, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av.y, bv[m].y, acc1, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av.z, bv[m].z, acc1, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av.w, bv[m].w, acc1, 0, 0, 0);
                }
            }
        }
        acc += acc1;
        nr += __shfl_xor(nr, 32, 64);
        const float inv = nr > 0.f ? 1.0f / sqrtf(nr) : 0.f;
        const float nx = nr > 0.f ? 1.f : 0.f;
        // lane (x, h) holds query i = 8 (r / 4) + 4 h + r % 4 against row x
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r / 4) + 4 * h + (r % 4);
            const int q = qb * 32 + i;
            float d2 = s_qn2[q] + nx - 2.f * acc[r] * inv;
            d2 = d2 > 0.f ? d2 : 0.f;
            const bool ok = row_ok && s_qid[q] >= 0 && row != (int64_t)s_qid[q];
            const uint64_t key =
                ok ? (((uint64_t)__float_as_uint(d2) << 32) | (uint64_t)row) : kNoKey;
            if (key < s_thr[w][i]) {
                const uint32_t pos = atomicAdd(&s_cnt[w][i], 1u);
                s_stage[w][i][pos] = key;  // pos < 32: one row per lane x
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        __builtin_amdgcn_wave_barrier();
        if (h == 0) {
            const uint32_t c = s_cnt[w][x];
            if (c > 0u) {
                uint64_t* L = s_list[w][x];
                uint32_t len = s_len[w][x];
                for (uint32_t e = 0; e < c; ++e) {
                    const uint64_t key = s_stage[w][x][e];
                    if (len == (uint32_t)k && key >= L[k - 1]) continue;
                    int p = len < (uint32_t)k ? (int)len : k - 1;
                    while (p > 0 && L[p - 1] > key) {
                        L[p] = L[p - 1];
                        --p;
                    }
                    L[p] = key;
                    if (len < (uint32_t)k) ++len;
                }
                s_len[w][x] = len;
                s_cnt[w][x] = 0u;
                s_thr[w][x] = len == (uint32_t)k ? L[k - 1] : kNoKey;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        __builtin_amdgcn_wave_barrier();
    }
    if (h == 0) {
        const uint32_t len = s_len[w][x];
        uint64_t* dst = A.partial + ((size_t)S * A.nqp + qb * 32 + x) * k;
        for (int t = 0; t < k; ++t) dst[t] = (uint32_t)t < len ? s_list[w][x][t] : kNoKey;
    }
}

// The k smallest keys of query q over all NS lists: running best k plus a
// chunk of candidates, bitonic-sorted together in LDS.
__global__ __launch_bounds__(kBlock) void k_knn_merge(const uint64_t* __restrict__ partial,
                                                      int64_t NS, int32_t nqp, int32_t k,
                                                      int32_t q_first, int32_t* __restrict__ ids,
                                                      float* __restrict__ dist,
                                                      const int32_t* __restrict__ gate) {
    __shared__ uint64_t s_buf[kKnnMergeCap];
    if (gate && *gate == 0) return;
    const int q = blockIdx.x;
    const int64_t total = NS * k;
    for (int i = threadIdx.x; i < k; i += kBlock) s_buf[i] = kNoKey;
    for (int64_t base = 0; base < total; base += kKnnMergeCap - k) {
        const int64_t chunk =
            total - base < kKnnMergeCap - k ? total - base : (int64_t)(kKnnMergeCap - k);
        for (int i = threadIdx.x; i < kKnnMergeCap - k; i += kBlock) {
            uint64_t v = kNoKey;
            if (i < chunk) {
                const int64_t c = base + i;
                v = partial[((c / k) * nqp + q) * k + (c % k)];
            }
            s_buf[k + i] = v;
        }
        __syncthreads();
        for (int size = 2; size <= kKnnMergeCap; size <<= 1) {
            for (int st = size >> 1; st > 0; st >>= 1) {
                for (int i = threadIdx.x; i < kKnnMergeCap / 2; i += kBlock) {
                    const int lo = 2 * i - (i & (st - 1));
                    const int hi = lo + st;
                    const bool up = (lo & size) == 0;
                    const uint64_t a = s_buf[lo], b = s_buf[hi];
                    if ((a > b) == up) {
                        s_buf[lo] = b;
                        s_buf[hi] = a;
                    }
                }
                __syncthreads();
            }
        }
    }
    for (int t = threadIdx.x; t < k; t += kBlock) {
        const uint64_t key = s_buf[t];
        const int64_t o = (int64_t)(q_first + q) * k + t;
        ids[o] = key == kNoKey ? -1 : (int32_t)(uint32_t)key;
        dist[o] = key == kNoKey ? __builtin_nanf("") : sqrtf(__uint_as_float((uint32_t)(key >> 32)));
    }
}

// The same search for dim <= 128 on the fp16 matrix cores.  Queries and rows
// are normalised and scaled by 2^10 (|x| <= 1024), and each value is split
// into two fp16 parts, x = hi + lo + e with |e| <= 2^-22 |x| (hi the nearest
// fp16 of x, lo that of the exact remainder x - hi); the three products
// hi.hi + hi.lo + lo.hi (v_mfma_f32_32x32x16_f16, exact fp16 products summed
// in fp32) leave out lo.lo and e, about 2^-21 of each term, against the 2^-24
// of fp32 products: well inside the search's distance bound.  A 16-dimension
// chunk takes three matrix instructions here against eight in fp32.
// Operand layout (checked on the GPU): A[i][c] comes from element c % 8 of
// lane i + 32 (c / 8), B[c][j] from element c % 8 of lane j + 32 (c / 8); the
// accumulators are laid out as for the fp32 instruction.
typedef _Float16 knn_h8 __attribute__((ext_vector_type(8)));
constexpr float kKnnSplitScale = 1024.0f;                  // 2^10
constexpr float kKnnSplitUnscale = 1.0f / (1024.0f * 1024.0f);  // 2^-20, exact

// The split of 8 values scaled by sc.  Each product v is pinned as one fp32
// value (an empty asm statement that the compiler must assume redefines it),
// so the multiplication cannot be fused into the conversions: hi is the fp16
// of v and the remainder v - hi is exact, so hi + lo equals v up to the
// rounding of lo.  Left to the default contraction, the product was rounded
// once for hi and once, differently, for lo, and at an exact fp16 tie hi + lo
// missed v by one fp16 step; the pinned form also measured faster than
// placing hi on the fp16 grid with integer operations on the bits of v.
__device__ __forceinline__ void knn_split8(float4 a, float4 b, float sc, knn_h8& hi,
                                           knn_h8& lo) {
    float v[8] = {a.x * sc, a.y * sc, a.z * sc, a.w * sc, b.x * sc, b.y * sc, b.z * sc,
                  b.w * sc};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        asm volatile("" : "+v"(v[e]));
        const _Float16 h = (_Float16)v[e];
        hi[e] = h;
        lo[e] = (_Float16)(v[e] - (float)h);
    }
}

// The hi parts alone of knn_split8 (the same pinned products, the same
// conversions): hi[e] equals knn_split8's hi[e] bit for bit.
__device__ __forceinline__ knn_h8 knn_hi8(float4 a, float4 b, float sc) {
    float v[8] = {a.x * sc, a.y * sc, a.z * sc, a.w * sc, b.x * sc, b.y * sc, b.z * sc,
                  b.w * sc};
    knn_h8 hi;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        asm volatile("" : "+v"(v[e]));
        hi[e] = (_Float16)v[e];
    }
    return hi;
}

// Squared norm of the 16 values v[0 .. 3] in a fixed order of explicit fused
// multiply-adds, and that of a row held by a lane pair (x, 0), (x, 1) as
// 16 float4 each: four such sums per lane, each added to its partner's, then
// (P0 + P1) + (P2 + P3).  Every fp16 search forms a row's norm this way (the
// four-block search from partial sums that its four waves exchange), so all of
// them compute the same scale and the same distances for a row.
__device__ __forceinline__ float knn_sq4(const float4* v) {
    float p = 0.f;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        float t = v[m].x * v[m].x;
        t = fmaf(v[m].y, v[m].y, t);
        t = fmaf(v[m].z, v[m].z, t);
        t = fmaf(v[m].w, v[m].w, t);
        p += t;
    }
    return p;
}

__device__ __forceinline__ float knn_row_norm(const float4 (&v)[16]) {
    float P[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        P[i] = knn_sq4(v + 4 * i);
        P[i] += __shfl_xor(P[i], 32, 64);
    }
    return (P[0] + P[1]) + (P[2] + P[3]);
}

__global__ __launch_bounds__(kKnnWavesR * 64) void k_knn_tiles_h(KnnArgs A) {
    __shared__ uint64_t s_list[kKnnWavesR][32][kKnnMaxK];
    __shared__ uint64_t s_stage[kKnnWavesR][32][32];
    __shared__ uint64_t s_thr[kKnnWavesR][32];
    __shared__ uint32_t s_cnt[kKnnWavesR][32];
    __shared__ uint32_t s_len[kKnnWavesR][32];

    if (A.gate && *A.gate == 0) return;  // the threshold scans answered every query
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int x = lane & 31, h = lane >> 5;
    const int D = A.D, k = A.k;
    const int qb = w % A.QB;
    const int wpb = kKnnWavesR / A.QB;
    const int64_t S = (int64_t)blockIdx.x * wpb + w / A.QB;
    const int64_t NS = (int64_t)gridDim.x * wpb;
    constexpr int kCh = kKnnDimChunk / 16;  // 16-dimension chunks
    // lane (x, h) holds dimensions 16 s + 8 h .. 16 s + 8 h + 7 of chunk s
    const int d0 = 8 * h;

    // operands of query qb * 32 + x (already normalised)
    knn_h8 qh[kCh], ql[kCh];
    {
        const float* qrow = A.qn + (int64_t)(qb * 32 + x) * D;
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            const int d = 16 * c + d0;
            const float4 a = d + 4 <= D ? *reinterpret_cast<const float4*>(qrow + d)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
            const float4 b = d + 8 <= D ? *reinterpret_cast<const float4*>(qrow + d + 4)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
            knn_split8(a, b, kKnnSplitScale, qh[c], ql[c]);
        }
    }
    // this lane's 16 score slots: query i = 8 (r / 4) + 4 h + r % 4; the
    // squared norm of a normalised query is 1 (0 for a zero query): one bit.
    // A padding slot (no query) keeps the threshold -inf: nothing passes it.
    float thr[16];
    int32_t qid[16];
    uint32_t qone = 0u;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int q = qb * 32 + 8 * (r / 4) + 4 * h + (r % 4);
        qone |= A.qn2[q] > 0.f ? 1u << r : 0u;
        qid[r] = A.qid[q];
        thr[r] = qid[r] >= 0 ? __builtin_inff() : -__builtin_inff();
    }
    if (lane < 32) {
        s_thr[w][lane] = kNoKey;
        s_cnt[w][lane] = 0u;
        s_len[w][lane] = 0u;
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    __builtin_amdgcn_wave_barrier();

    for (int64_t t = S; t < A.tiles; t += NS) {
        const int64_t row = t * 32 + x;
        const bool ok = row < A.N;
        const float* src = A.T + (ok ? row : 0) * (int64_t)D;
        float4 bv[2 * kCh];
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            const int d = 16 * c + d0;
            bv[2 * c] = (ok && d + 4 <= D) ? *reinterpret_cast<const float4*>(src + d)
                                           : make_float4(0.f, 0.f, 0.f, 0.f);
            bv[2 * c + 1] = (ok && d + 8 <= D) ? *reinterpret_cast<const float4*>(src + d + 4)
                                               : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        const float nr = knn_row_norm(bv);
        const float sc = nr > 0.f ? kKnnSplitScale / sqrtf(nr) : 0.f;
        const float nx = nr > 0.f ? 1.f : 0.f;
        knn_acc16 acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                         0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            knn_h8 bh, bl;
            knn_split8(bv[2 * c], bv[2 * c + 1], sc, bh, bl);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(qh[c], bh, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(qh[c], bl, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ql[c], bh, acc, 0, 0, 0);
        }
        bool staged = false;
        const float nx1 = nx + 1.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            // d^2 = |q|^2 + [r != 0] - 2 <q, r>, clamped at 0
            const float base = (qone >> r) & 1u ? nx1 : nx;
            float d2 = fmaf(-2.f * kKnnSplitUnscale, acc[r], base);
            d2 = d2 > 0.f ? d2 : 0.f;
            if (d2 <= thr[r] && ok && row != (int64_t)qid[r]) {
                const int i = 8 * (r / 4) + 4 * h + (r % 4);
                const uint64_t key = ((uint64_t)__float_as_uint(d2) << 32) | (uint64_t)row;
                if (key < s_thr[w][i]) {
                    const uint32_t pos = atomicAdd(&s_cnt[w][i], 1u);
                    s_stage[w][i][pos] = key;  // pos < 32: one row per lane x
                    staged = true;
                }
            }
        }
        if (__ballot(staged) == 0ull) continue;  // wave-uniform: nothing to merge
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        __builtin_amdgcn_wave_barrier();
        if (h == 0) {
            const uint32_t c = s_cnt[w][x];
            if (c > 0u) {
                uint64_t* L = s_list[w][x];
                uint32_t len = s_len[w][x];
                for (uint32_t e = 0; e < c; ++e) {
                    const uint64_t key = s_stage[w][x][e];
                    if (len == (uint32_t)k && key >= L[k - 1]) continue;
                    int p = len < (uint32_t)k ? (int)len : k - 1;
                    while (p > 0 && L[p - 1] > key) {
                        L[p] = L[p - 1];
                        --p;
                    }
                    L[p] = key;
                    if (len < (uint32_t)k) ++len;
                }
                s_len[w][x] = len;
                s_cnt[w][x] = 0u;
                s_thr[w][x] = len == (uint32_t)k ? L[k - 1] : kNoKey;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r / 4) + 4 * h + (r % 4);
            const uint64_t tk = s_thr[w][i];
            const float tv = tk == kNoKey ? __builtin_inff() : __uint_as_float((uint32_t)(tk >> 32));
            thr[r] = qid[r] >= 0 ? tv : -__builtin_inff();
        }
    }
    if (h == 0) {
        const uint32_t len = s_len[w][x];
        uint64_t* dst = A.partial + ((size_t)S * A.nqp + qb * 32 + x) * k;
        for (int t = 0; t < k; ++t) dst[t] = (uint32_t)t < len ? s_list[w][x][t] : kNoKey;
    }
}

// The same search when a pass holds four query blocks (97-128 queries): the
// four waves of a row tile (one per query block) share its load, norm and
// split instead of each doing all of it.  Wave qb loads chunks 2 qb and
// 2 qb + 1 (16-dimension chunks) of the tile's rows and publishes their
// partial squared norms; after a barrier each wave forms the row scales,
// splits its two chunks and publishes the fp16 parts; after a second barrier
// every wave reads all eight chunks' parts from LDS for its products.  Every
// wave of the workgroup runs the same number of iterations (that of the
// workgroup's first tile stream; a stream past its last tile loads nothing
// and offers no candidates), so all of them reach both barriers each time.
// Candidates are staged as (d^2, row in tile) to leave LDS for the parts.
__global__ __launch_bounds__(kKnnWavesR * 64) void k_knn_tiles_h4(KnnArgs A) {
    constexpr int kQB = 4;
    constexpr int kStreams = kKnnWavesR / kQB;  // tile streams per workgroup
    constexpr int kCh = kKnnDimChunk / 16;      // 16-dimension chunks
    __shared__ uint64_t s_list[kKnnWavesR][32][kKnnMaxK];
    __shared__ float s_sd[kKnnWavesR][32][32];    // staged d^2
    __shared__ uint8_t s_sx[kKnnWavesR][32][32];  // staged row within the tile
    __shared__ uint64_t s_thr[kKnnWavesR][32];
    __shared__ uint32_t s_cnt[kKnnWavesR][32];
    __shared__ uint32_t s_len[kKnnWavesR][32];
    __shared__ float s_nr[kStreams][kQB][32];     // partial squared norms of the rows
    // fp16 parts of the tile: [stream][chunk][row][h] = {hi, lo} of 8 dimensions
    __shared__ knn_h8 s_part[kStreams][kCh][32][2][2];

    if (A.gate && *A.gate == 0) return;  // the threshold scans answered every query
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int x = lane & 31, h = lane >> 5;
    const int D = A.D, k = A.k;
    const int qb = w % kQB;
    const int st = w / kQB;
    const int64_t S0 = (int64_t)blockIdx.x * kStreams;
    const int64_t S = S0 + st;
    const int64_t NS = (int64_t)gridDim.x * kStreams;
    const int d0 = 8 * h;
    // iterations of every wave: those of the workgroup's first stream
    const int64_t iters = A.tiles > S0 ? (A.tiles - S0 + NS - 1) / NS : 0;

    // operands of query qb * 32 + x (already normalised)
    knn_h8 qh[kCh], ql[kCh];
    {
        const float* qrow = A.qn + (int64_t)(qb * 32 + x) * D;
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            const int d = 16 * c + d0;
            const float4 a = d + 4 <= D ? *reinterpret_cast<const float4*>(qrow + d)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
            const float4 b = d + 8 <= D ? *reinterpret_cast<const float4*>(qrow + d + 4)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
            knn_split8(a, b, kKnnSplitScale, qh[c], ql[c]);
        }
    }
    float thr[16];
    int32_t qid[16];
    uint32_t qone = 0u;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int q = qb * 32 + 8 * (r / 4) + 4 * h + (r % 4);
        qone |= A.qn2[q] > 0.f ? 1u << r : 0u;
        qid[r] = A.qid[q];
        thr[r] = qid[r] >= 0 ? __builtin_inff() : -__builtin_inff();
    }
    if (lane < 32) {
        s_thr[w][lane] = kNoKey;
        s_cnt[w][lane] = 0u;
        s_len[w][lane] = 0u;
    }

    // this wave's two chunks of row x of its stream's tile of iteration it2
    // (zeros past the table)
    auto load_chunks = [&](int64_t it2, float4 (&dst)[4]) {
        const int64_t t2 = S + it2 * NS;
        const int64_t row2 = t2 * 32 + x;
        const bool ok2 = it2 < iters && t2 < A.tiles && row2 < A.N;
        const float* src = A.T + (ok2 ? row2 : 0) * (int64_t)D;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int d = 16 * (2 * qb + j) + d0;
            dst[2 * j] = (ok2 && d + 4 <= D) ? *reinterpret_cast<const float4*>(src + d)
                                             : make_float4(0.f, 0.f, 0.f, 0.f);
            dst[2 * j + 1] = (ok2 && d + 8 <= D) ? *reinterpret_cast<const float4*>(src + d + 4)
                                                 : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    // The chunks are loaded one iteration ahead: the next tile's loads are in
    // flight during the products and the candidate merge of the current one
    // (the barriers wait for LDS accesses only; loading two tiles ahead, in
    // two register buffers, measured no faster).
    float4 nb[4];
    load_chunks(0, nb);

    for (int64_t it = 0; it < iters; ++it) {
        const int64_t t = S + it * NS;
        const int64_t row = t * 32 + x;
        const bool ok = t < A.tiles && row < A.N;
        float4 bv[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) bv[m] = nb[m];
        float pn = knn_sq4(bv);
        pn += __shfl_xor(pn, 32, 64);
        if (h == 0) s_nr[st][qb][x] = pn;
        __syncthreads();
        const float nr = (s_nr[st][0][x] + s_nr[st][1][x]) + (s_nr[st][2][x] + s_nr[st][3][x]);
        const float sc = nr > 0.f ? kKnnSplitScale / sqrtf(nr) : 0.f;
        const float nx = nr > 0.f ? 1.f : 0.f;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            knn_h8 bh, bl;
            knn_split8(bv[2 * j], bv[2 * j + 1], sc, bh, bl);
            s_part[st][2 * qb + j][x][h][0] = bh;
            s_part[st][2 * qb + j][x][h][1] = bl;
        }
        load_chunks(it + 1, nb);
        __syncthreads();
        knn_acc16 acc = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                         0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            const knn_h8 bh = s_part[st][c][x][h][0];
            const knn_h8 bl = s_part[st][c][x][h][1];
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(qh[c], bh, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(qh[c], bl, acc, 0, 0, 0);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ql[c], bh, acc, 0, 0, 0);
        }
        bool staged = false;
        const float nx1 = nx + 1.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            // d^2 = |q|^2 + [r != 0] - 2 <q, r>, clamped at 0
            const float base = (qone >> r) & 1u ? nx1 : nx;
            float d2 = fmaf(-2.f * kKnnSplitUnscale, acc[r], base);
            d2 = d2 > 0.f ? d2 : 0.f;
            if (d2 <= thr[r] && ok && row != (int64_t)qid[r]) {
                const int i = 8 * (r / 4) + 4 * h + (r % 4);
                const uint64_t key = ((uint64_t)__float_as_uint(d2) << 32) | (uint64_t)row;
                if (key < s_thr[w][i]) {
                    const uint32_t pos = atomicAdd(&s_cnt[w][i], 1u);
                    s_sd[w][i][pos] = d2;  // pos < 32: one row per lane x
                    s_sx[w][i][pos] = (uint8_t)x;
                    staged = true;
                }
            }
        }
        if (__ballot(staged) == 0ull) continue;  // wave-uniform: nothing to merge
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        __builtin_amdgcn_wave_barrier();
        if (h == 0) {
            const uint32_t c = s_cnt[w][x];
            if (c > 0u) {
                uint64_t* L = s_list[w][x];
                uint32_t len = s_len[w][x];
                for (uint32_t e = 0; e < c; ++e) {
                    const uint64_t key = ((uint64_t)__float_as_uint(s_sd[w][x][e]) << 32) |
                                         (uint64_t)(t * 32 + s_sx[w][x][e]);
                    if (len == (uint32_t)k && key >= L[k - 1]) continue;
                    int p = len < (uint32_t)k ? (int)len : k - 1;
                    while (p > 0 && L[p - 1] > key) {
                        L[p] = L[p - 1];
                        --p;
                    }
                    L[p] = key;
                    if (len < (uint32_t)k) ++len;
                }
                s_len[w][x] = len;
                s_cnt[w][x] = 0u;
                s_thr[w][x] = len == (uint32_t)k ? L[k - 1] : kNoKey;
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int i = 8 * (r / 4) + 4 * h + (r % 4);
            const uint64_t tk = s_thr[w][i];
            const float tv = tk == kNoKey ? __builtin_inff() : __uint_as_float((uint32_t)(tk >> 32));
            thr[r] = qid[r] >= 0 ? tv : -__builtin_inff();
        }
    }
    if (h == 0) {
        const uint32_t len = s_len[w][x];
        uint64_t* dst = A.partial + ((size_t)S * A.nqp + qb * 32 + x) * k;
        for (int t = 0; t < k; ++t) dst[t] = (uint32_t)t < len ? s_list[w][x][t] : kNoKey;
    }
}

// ---------------------------------------------------------------------------
// Threshold scans (dim <= 128): the default search.  A scan visits the row
// tiles i * step (0 <= i < count); every wave takes whole 32-row tiles, loads
// the next one while it works on the current one, and forms the distances of
// its tile to every query of the pass with the fp16 parts of the queries in
// LDS.  Row x's norm, scale and split, the products and d^2 are those of the
// list-merging kernels above, bit for bit (the matrix instruction takes the
// row parts as its first operand here, the same products in the same order).
// A (row, query) pair whose d^2 is at most the query's bound tau is appended
// to the query's candidate list; only the count of a list that overflows its
// capacity keeps growing.  Between scans a selection sorts each list: its
// k-th key bounds the k-th distance over the whole table (any k rows do), so
// the next, denser scan keeps every row of the true answer.  The scans are
// nested (each one's tiles are among the next one's), so each finds at least
// the k rows that set its bound; the last one visits every tile and its k
// smallest keys are the answer.
// A tile is screened first by the hi.hi products alone (one matrix
// instruction per chunk instead of three, no lo parts): they differ from the
// full products hi.hi + hi.lo + lo.hi by at most the dropped terms,
// sum |hi_q lo_r| + |lo_q hi_r| <= 2^-10 (1 + 2^-10) 2^20 with |q|, |r| <= 2^10
// after scaling, plus the accumulations' roundings (at most 384 of 2^-4
// each) and fp16 subnormal steps: below 1100 units of the product.  For a
// present, nonzero row, d^2 <= tau needs acc >= (|q|^2 + 1 - tau) 2^19 - 2
// (the bound is computed within 2^-3 and d^2's one rounding moves it by at
// most 2^-21, a quarter of a unit of acc), so a screened product below that
// less kKnnScreenMargin = 1536 clears the pair.  A query block with any pair
// left, or a tile with a zero or missing row, gets the full products of the
// list search (bit for bit) and the exact test.
// ---------------------------------------------------------------------------
struct KnnScanArgs {
    const float* T;
    int64_t N;
    int32_t D;
    int32_t cap;    // keys kept per list
    int64_t step;   // tiles i * step, 0 <= i < count
    int64_t count;
    const float* qn;
    const float* qn2;
    const int32_t* qid;
    const float* tau;
    uint32_t* cnt;
    uint64_t* cand;  // [query slot][cap]
};

constexpr float kKnnAccPerD2 = 524288.0f;  // 2^19: a unit of d^2 in the product's units
constexpr float kKnnScreenMargin = 1536.0f;  // product units: hi.hi against the full products

// The exact test of a tile's pairs with query block qb and the append of the
// passing ones (a tile with a candidate, a zero or a missing row).
template <int QB>
__device__ __forceinline__ void knn_scan_append(const KnnScanArgs& A, int qb, int x, int h,
                                                int64_t t, uint64_t live,
                                                const knn_acc16& acc) {
    const int q = qb * 32 + x;
    const float tau = A.tau[q];
    const int64_t qid = A.qid[q];
    const bool q1 = A.qn2[q] > 0.f;
    const int64_t rows = A.N - t * 32;  // rows of the tile present
    uint32_t pass = 0u;
    float d2v[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        // d^2 = |q|^2 + [row != 0] - 2 <q, row>, clamped at 0
        const int m = 8 * (r / 4) + 4 * h + (r % 4);
        const float nx = (live >> m) & 1ull ? 1.f : 0.f;
        const float base = q1 ? nx + 1.f : nx;
        float d2 = fmaf(-2.f * kKnnSplitUnscale, acc[r], base);
        d2 = d2 > 0.f ? d2 : 0.f;
        d2v[r] = d2;
        if (d2 <= tau && m < rows && t * 32 + m != qid) pass |= 1u << r;
    }
    if (pass == 0u) return;
    uint32_t pos = atomicAdd(&A.cnt[q], (uint32_t)__popc(pass));
    uint64_t* dst = A.cand + (size_t)q * A.cap;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        if (!((pass >> r) & 1u)) continue;
        const int m = 8 * (r / 4) + 4 * h + (r % 4);
        if (pos < (uint32_t)A.cap)
            dst[pos] = ((uint64_t)__float_as_uint(d2v[r]) << 32) | (uint64_t)(t * 32 + m);
        ++pos;
    }
}

// FULL: dim is 128, so no dimension of a chunk lies past the row.
template <int QB, bool FULL>
__global__ __launch_bounds__(kKnnScanWaves * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_knn_scan(KnnScanArgs A) {
    constexpr int kCh = kKnnDimChunk / 16;  // 16-dimension chunks
    // B operands: lane (x, h) of s_q[qb][c][p] holds the fp16 part p (0 hi,
    // 1 lo) of query qb * 32 + x's dimensions 16 c + 8 h .. 16 c + 8 h + 7
    __shared__ knn_h8 s_q[QB][kCh][2][64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int x = lane & 31, h = lane >> 5;
    const int D = A.D;
    const int d0 = 8 * h;
    for (int j = w; j < QB * kCh; j += kKnnScanWaves) {
        const int qb = j / kCh, c = j % kCh;
        const float* qrow = A.qn + (int64_t)(qb * 32 + x) * D;
        const int d = 16 * c + d0;
        const float4 a = d + 4 <= D ? *reinterpret_cast<const float4*>(qrow + d)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 b = d + 8 <= D ? *reinterpret_cast<const float4*>(qrow + d + 4)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
        knn_h8 hi, lo;
        knn_split8(a, b, kKnnSplitScale, hi, lo);
        s_q[qb][c][0][lane] = hi;
        s_q[qb][c][1][lane] = lo;
    }
    // lane (x, h) holds query qb * 32 + x of every block against rows
    // 8 (r / 4) + 4 h + r % 4 of the tile (accumulator r); a screened
    // product below athr[qb] is no candidate for a present, nonzero row
    float athr[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
        const int q = qb * 32 + x;
        const float q1 = A.qn2[q] > 0.f ? 1.f : 0.f;
        athr[qb] = ((q1 + 1.f) - A.tau[q]) * kKnnAccPerD2 - 2.f - kKnnScreenMargin;
    }
    __syncthreads();

    const int64_t W = (int64_t)gridDim.x * kKnnScanWaves;
    const int64_t i0 = (int64_t)blockIdx.x * kKnnScanWaves + w;
    // Row x of tile i * step: lane (x, h) loads dimensions 16 c + 8 h .. + 7
    // of every chunk c.  Past the scan's last tile or the table a lane loads
    // row 0 instead (its rows are marked missing below); past dim, zeros.
    auto load_tile = [&](int64_t i, float4 (&dst)[2 * kCh]) {
        const int64_t row = i * A.step * 32 + x;
        const bool ok = i < A.count && row < A.N;
        const float* src = A.T + (ok ? row : 0) * (int64_t)D;
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            const int d = 16 * c + d0;
            if (FULL) {
                dst[2 * c] = *reinterpret_cast<const float4*>(src + d);
                dst[2 * c + 1] = *reinterpret_cast<const float4*>(src + d + 4);
            } else {
                dst[2 * c] = d + 4 <= D ? *reinterpret_cast<const float4*>(src + d)
                                        : make_float4(0.f, 0.f, 0.f, 0.f);
                dst[2 * c + 1] = d + 8 <= D ? *reinterpret_cast<const float4*>(src + d + 4)
                                            : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
    };
    auto scan_tile = [&](int64_t i, const float4 (&bv)[2 * kCh]) {
        const int64_t t = i * A.step;
        const float nr = knn_row_norm(bv);
        const float sc = nr > 0.f ? kKnnSplitScale / sqrtf(nr) : 0.f;
        // bit m (and m + 32): row m of the tile is present and nonzero
        const uint64_t live = __ballot(nr > 0.f && t * 32 + x < A.N);
        // the screen: hi.hi products of every query block
        knn_acc16 acc[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[qb][r] = 0.f;
#pragma unroll
        for (int c = 0; c < kCh; ++c) {
            const knn_h8 bh = knn_hi8(bv[2 * c], bv[2 * c + 1], sc);
#pragma unroll
            for (int qb = 0; qb < QB; ++qb)
                acc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(bh, s_q[qb][c][0][lane],
                                                                 acc[qb], 0, 0, 0);
        }
        // bit qb: the block has a pair left (wave-uniform)
        uint32_t need = 0u;
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
            bool look = live != ~0ull;
#pragma unroll
            for (int r = 0; r < 16; ++r) look |= acc[qb][r] >= athr[qb];
            need |= __ballot(look) != 0ull ? 1u << qb : 0u;
        }
        // the full products of the list search for those blocks, then the exact test
#pragma unroll 1
        for (; need != 0u; need &= need - 1u) {
            const int qb = __builtin_ctz(need);
            knn_acc16 ex = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f,
                            0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < kCh; ++c) {
                knn_h8 bh, bl;
                knn_split8(bv[2 * c], bv[2 * c + 1], sc, bh, bl);
                const knn_h8 qh = s_q[qb][c][0][lane];
                const knn_h8 ql = s_q[qb][c][1][lane];
                ex = __builtin_amdgcn_mfma_f32_32x32x16_f16(bh, qh, ex, 0, 0, 0);
                ex = __builtin_amdgcn_mfma_f32_32x32x16_f16(bl, qh, ex, 0, 0, 0);
                ex = __builtin_amdgcn_mfma_f32_32x32x16_f16(bh, ql, ex, 0, 0, 0);
            }
            knn_scan_append<QB>(A, qb, x, h, t, live, ex);
        }
    };
    // two register buffers in turn: a tile's rows load during the previous
    // tile's products
    float4 ba[2 * kCh], bb[2 * kCh];
    load_tile(i0, ba);
    for (int64_t i = i0; i < A.count; i += 2 * W) {
        load_tile(i + W, bb);
        scan_tile(i, ba);
        if (i + W >= A.count) break;
        load_tile(i + 2 * W, ba);
        scan_tile(i + W, bb);
    }
}

// Candidate selection, one workgroup per query slot: the list's kept keys
// (at most cap, a power of two) sorted in LDS by a bitonic network.  After a
// sample scan the k-th key's d^2 becomes the query's bound (fewer than k keys
// leave it); after the last scan the k smallest keys are the answer, written
// as the list-merging search writes it, and a list that overflowed opens the
// gate for that search.  The count is reset for the next scan.
struct KnnSelectArgs {
    uint32_t* cnt;
    const uint64_t* cand;
    int32_t cap;
    int32_t k;
    int32_t last;      // 1: the last scan
    int32_t m;         // queries of the pass (slots beyond are padding)
    int32_t q_first;   // the pass's first query
    float* tau;
    int32_t* ids;
    float* dist;
    int32_t* gate;
};

__global__ __launch_bounds__(kKnnSelectThreads) void k_knn_select(KnnSelectArgs S) {
    extern __shared__ uint64_t s_key[];
    const int q = blockIdx.x, tid = threadIdx.x;
    const uint32_t c = S.cnt[q];
    const uint32_t n = c < (uint32_t)S.cap ? c : (uint32_t)S.cap;
    uint32_t P = 2u;
    while (P < n) P <<= 1;
    for (uint32_t i = tid; i < P; i += kKnnSelectThreads)
        s_key[i] = i < n ? S.cand[(size_t)q * S.cap + i] : kNoKey;
    __syncthreads();
    for (uint32_t size = 2; size <= P; size <<= 1) {
        for (uint32_t st = size >> 1; st > 0; st >>= 1) {
            for (uint32_t i = tid; i < P / 2; i += kKnnSelectThreads) {
                const uint32_t lo = 2 * i - (i & (st - 1));
                const uint32_t hi = lo + st;
                const bool up = (lo & size) == 0;
                const uint64_t a = s_key[lo], b = s_key[hi];
                if ((a > b) == up) {
                    s_key[lo] = b;
                    s_key[hi] = a;
                }
            }
            __syncthreads();
        }
    }
    if (S.last) {
        if (q < S.m) {
            for (int t = tid; t < S.k; t += kKnnSelectThreads) {
                const uint64_t key = (uint32_t)t < P ? s_key[t] : kNoKey;
                const int64_t o = (int64_t)(S.q_first + q) * S.k + t;
                S.ids[o] = key == kNoKey ? -1 : (int32_t)(uint32_t)key;
                S.dist[o] = key == kNoKey ? __builtin_nanf("")
                                          : sqrtf(__uint_as_float((uint32_t)(key >> 32)));
            }
        }
        if (tid == 0 && c > (uint32_t)S.cap) *S.gate = 1;
    } else if (tid == 0 && n >= (uint32_t)S.k) {
        S.tau[q] = __uint_as_float((uint32_t)(s_key[S.k - 1] >> 32));
    }
    if (tid == 0) S.cnt[q] = 0u;
}

int knn_pass_queries(int D) {
    int qp = kKnnQueryFloats / (D + 4);
    qp = qp > kKnnPass ? kKnnPass : qp;
    return (qp / 32) * 32;
}

// Lists of one pass: (workgroups) x (waves per query block).
int64_t knn_lists(int64_t N, int D, int QB) {
    const int64_t tiles = (N + 31) / 32;
    const int waves = D <= kKnnDimChunk ? kKnnWavesR : kKnnWaves;
    const int wpb = waves / QB;
    int64_t grid = (tiles + wpb - 1) / wpb;
    grid = grid < kKnnGrid ? grid : kKnnGrid;
    return grid * wpb;
}

template <int QB>
static void launch_knn_scan(const KnnScanArgs& A, hipStream_t s) {
    int64_t grid = (A.count + kKnnScanWaves - 1) / kKnnScanWaves;
    grid = grid < kKnnScanGrid ? grid : kKnnScanGrid;
    if (A.D == kKnnDimChunk)
        hipLaunchKernelGGL((k_knn_scan<QB, true>), dim3((unsigned)grid),
                           dim3(kKnnScanWaves * 64), 0, s, A);
    else
        hipLaunchKernelGGL((k_knn_scan<QB, false>), dim3((unsigned)grid),
                           dim3(kKnnScanWaves * 64), 0, s, A);
}

// Tile strides of the threshold scans, coarsest first: the first visits at
// most kKnnStageTiles tiles with no bound (so its lists cannot overflow), each
// next one a stride kKnnStageGrowth times finer, the last every tile.  Returns
// the number of scans.
int knn_scan_steps(int64_t tiles, int64_t* steps) {
    int64_t s = 1;
    while ((tiles + s - 1) / s > kKnnStageTiles) s *= kKnnStageGrowth;
    int n = 0;
    for (; s >= 1; s /= kKnnStageGrowth) steps[n++] = s;
    return n;
}

hipError_t launch_knn(const float* T, int64_t N, int32_t D, const int32_t* q, int32_t nq,
                      int32_t k, int32_t* ids, float* dist, const KnnBuffers& B,
                      bool lists_only, int32_t* status, hipStream_t s) {
    const int qp = knn_pass_queries(D);
    if (qp < 32 || k < 1 || k > kKnnMaxK || N < 1) return hipErrorInvalidValue;
    const bool scans = D <= kKnnDimChunk && !lists_only;
    const int64_t tiles = (N + 31) / 32;
    for (int32_t q0 = 0; q0 < nq; q0 += qp) {
        const int32_t m = nq - q0 < qp ? nq - q0 : qp;
        int QB = (m + 31) / 32;
        if (QB == 3) QB = 4;
        const int32_t nqp = 32 * QB;
        hipLaunchKernelGGL(k_knn_queries, dim3((unsigned)nqp), dim3(kBlock), 0, s, T, N, D,
                           q + q0, m, nqp, B.qn, B.qn2, B.qid, scans ? B.tau : nullptr,
                           scans ? B.cnt : nullptr, scans ? B.gate : nullptr, status);
        if (scans) {
            KnnScanArgs SA;
            SA.T = T;
            SA.N = N;
            SA.D = D;
            SA.cap = kKnnCandCap;
            SA.qn = B.qn;
            SA.qn2 = B.qn2;
            SA.qid = B.qid;
            SA.tau = B.tau;
            SA.cnt = B.cnt;
            SA.cand = B.cand;
            KnnSelectArgs SS;
            SS.cnt = B.cnt;
            SS.cand = B.cand;
            SS.cap = kKnnCandCap;
            SS.k = k;
            SS.m = m;
            SS.q_first = q0;
            SS.tau = B.tau;
            SS.ids = ids;
            SS.dist = dist;
            SS.gate = B.gate;
            int64_t steps[16];
            const int ns = knn_scan_steps(tiles, steps);
            for (int j = 0; j < ns; ++j) {
                SA.step = steps[j];
                SA.count = (tiles + steps[j] - 1) / steps[j];
                if (QB == 4)
                    launch_knn_scan<4>(SA, s);
                else if (QB == 2)
                    launch_knn_scan<2>(SA, s);
                else
                    launch_knn_scan<1>(SA, s);
                SS.last = j == ns - 1;
                hipLaunchKernelGGL(k_knn_select, dim3((unsigned)nqp), dim3(kKnnSelectThreads),
                                   sizeof(uint64_t) * kKnnCandCap, s, SS);
            }
        }
        // the list-merging search: for wider rows always, else only where a
        // final candidate list overflowed (the gate; otherwise its kernels
        // return at once)
        KnnArgs A;
        A.T = T;
        A.N = N;
        A.D = D;
        A.k = k;
        A.nqp = nqp;
        A.QB = QB;
        A.stride = D + 4;
        A.tiles = tiles;
        A.qn = B.qn;
        A.qn2 = B.qn2;
        A.qid = B.qid;
        A.partial = B.partial;
        A.gate = scans ? B.gate : nullptr;
        const int64_t NS = knn_lists(N, D, QB);
        if (D <= kKnnDimChunk) {
            const int64_t grid = NS / (kKnnWavesR / QB);
            if (QB == 4)
                hipLaunchKernelGGL(k_knn_tiles_h4, dim3((unsigned)grid), dim3(kKnnWavesR * 64), 0,
                                   s, A);
            else
                hipLaunchKernelGGL(k_knn_tiles_h, dim3((unsigned)grid), dim3(kKnnWavesR * 64), 0,
                                   s, A);
        } else {
            const int64_t grid = NS / (kKnnWaves / QB);
            hipLaunchKernelGGL(k_knn_tiles, dim3((unsigned)grid), dim3(kKnnWaves * 64), 0, s, A);
        }
        hipLaunchKernelGGL(k_knn_merge, dim3((unsigned)m), dim3(kBlock), 0, s, B.partial, NS, nqp,
                           k, q0, ids, dist, A.gate);
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// recall@k(u) = |N(u) & S| / k, S = the query's k nearest rows (ids[q k ..]),
// N(u) = the ids of u's ascending list other than u.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void k_eval_recall(const int64_t* __restrict__ off,
                                                    const int32_t* __restrict__ nbr, int64_t N,
                                                    int64_t E, const int32_t* __restrict__ q,
                                                    const int32_t* __restrict__ ids, int32_t k,
                                                    double* __restrict__ out,
                                                    int32_t* __restrict__ status) {
    const int qi = blockIdx.x;
    const int t = threadIdx.x;
    const int32_t u = q[qi];
    bool found = false;
    bool bad = u < 0 || (int64_t)u >= N;
    int64_t b = 0, e = 0;
    if (!bad) {
        b = off[u];
        e = off[u + 1];
        bad = b < 0 || e < b || e > E;
    }
    if (!bad && t < k) {
        const int32_t id = ids[(int64_t)qi * k + t];
        found = id >= 0 && id != u && in_sorted_list(nbr, b, e, id);
    }
    const uint64_t m = __ballot(found);
    if (t == 0) {
        if (bad) eval_fail(status, -2);
        out[qi] = bad ? __builtin_nan("") : (double)__popcll(m) / (double)k;
    }
}

hipError_t launch_eval_recall(const int64_t* off, const int32_t* nbr, int64_t N, int64_t E,
                              const int32_t* q, int32_t nq, const int32_t* ids, int32_t k,
                              double* out, int32_t* status, hipStream_t s) {
    if (nq == 0) return hipSuccess;
    if (k < 1 || k > 64) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_eval_recall, dim3((unsigned)nq), dim3(64), 0, s, off, nbr, N, E, q, ids,
                       k, out, status);
    return hipGetLastError();
}

__global__ void k_eval_status_clear(int32_t* status) {
    if (threadIdx.x == 0 && blockIdx.x == 0) *status = 0;
}

hipError_t launch_eval_status_clear(int32_t* status, hipStream_t s) {
    hipLaunchKernelGGL(k_eval_status_clear, dim3(1), dim3(64), 0, s, status);
    return hipGetLastError();
}

// Keys of the distances: their float bit patterns (non-negative values and
// NaN order as unsigned integers: every NaN after every value).
__global__ __launch_bounds__(kBlock) void k_eval_keys(const float* __restrict__ d, int64_t n,
                                                      uint32_t* __restrict__ keys) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    const float x = d[i];
    keys[i] = x != x ? 0xFFFFFFFFu : __float_as_uint(x);
}

hipError_t launch_eval_keys(const float* d, int64_t n, uint32_t* keys, hipStream_t s) {
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(k_eval_keys, dim3((unsigned)((n + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                       s, d, n, keys);
    return hipGetLastError();
}

}  // namespace huge
