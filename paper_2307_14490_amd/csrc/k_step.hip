// The training step proper: for every positive, gather its rows, take the
// (1 + K) dot products, the loss and the coefficients, and update the rows
// (HUGE Sec. 3.3.2: gather, forward and gradient, aggregate, update).
//
// Rows that occur once in the batch are rewritten in place by the thread
// group that read them -- no other group reads them.  A row that occurs
// several times is left untouched here: each occurrence stores its
// contribution in the slot the grouping gave it (a row's slots are
// consecutive, in occurrence order), and the finish kernel sums them in that
// order and updates the row once, so every read sees pre-step values.
#include "common.hpp"
#include "device.hpp"
#include "dispatch.hpp"

namespace huge {

// Sum of one double per thread over the workgroup, written by thread 0.
__device__ __forceinline__ void block_loss(float loss, double* __restrict__ out) {
    __shared__ double s_w[kBlock / 64];
    double v = (double)loss;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    if ((threadIdx.x & 63) == 0) s_w[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        double acc = 0.0;
#pragma unroll
        for (int w = 0; w < kBlock / 64; ++w) acc += s_w[w];
        out[blockIdx.x] = acc;
    }
}

// NB negative rows are in flight at a time (NB = K up to 8, rounded up to
// a supported block): the block holds NB rows of registers, so a smaller one
// raises the occupancy, which the kernel needs to hide its memory latency.
// IO is the row policy of the tables (G lanes per row), DIO the same element
// ownership over the float contributions of repeated rows.  The context rows
// stay packed in registers (bf16: half the registers) and are widened where
// used; the source row and the source gradient are held widened.
// FULL: K == NB, the negatives are one block of compile-time size.
// Negative k of positive i is neg[i * neg_stride + k] (the sort keys in
// occurrence order, whose slots 2.. are the negatives' row ids).  info[o] is
// -1 for a row occurring once, else the occurrence's duplicate-buffer slot;
// the kernel sets every entry it finds >= 0 back to -1 once it has read it,
// so that the array is all -1 again for the next batch in this slot (the
// grouping writes only the repeated occurrences).
template <int G, int NB, bool FULL, typename IO, typename DIO>
__global__ __launch_bounds__(kBlock) void k_fused_step(TableArgs t, Control* __restrict__ ctl,
                                                       StepArgs a, const int32_t* __restrict__ neg,
                                                       uint32_t neg_stride,
                                                       int32_t* __restrict__ info,
                                                       float* __restrict__ dup,
                                                       double* __restrict__ lossp) {
    using E = typename IO::Elem;
    using Reg = typename IO::Reg;
    constexpr int C = IO::C;
    constexpr int R = IO::R;
    static_assert(DIO::C == C, "the contribution layout must match the row layout");
    // Registers: at least 88 VGPRs for float tables -- five waves per SIMD
    // (440 of 512 registers), not six -- and at least 104 for bf16 tables,
    // whose variants need more than 88: four waves, not five -- so that one
    // wave of a grouping kernel of the next batch (at most 72 VGPRs) fits
    // beside them on every SIMD.  The empty statement marks the register as
    // used; it generates no instruction.
    if constexpr (sizeof(E) == 2)
        asm volatile("" ::: "v103");
    else
        asm volatile("" ::: "v87");
    constexpr int PPB = kBlock / G;
    // A group of at least 1 + NB lanes evaluates its sigmoids and softplus
    // terms one value per lane instead of every lane evaluating all of them;
    // the positive's too where its row takes at most four registers (a wider
    // row would stay live until the first negatives' coefficients, which
    // costs more occupancy than the one evaluation saves).
    constexpr bool kLaneCoefs = G >= NB + 1;
    constexpr bool kLanePos = kLaneCoefs && sizeof(Reg) * R <= 16;
    const int grp = threadIdx.x / G;
    const int lane = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * PPB + grp;
    const int K = FULL ? NB : t.K;
    if (ctl->step_bad) {  // a no-op step: only the slots the grouping may have set
        if (i < a.n && lane == 0) {
            const uint32_t o = (uint32_t)i * (uint32_t)(2 + K);
            for (int q = 0; q < 2 + K; ++q)
                if (info[o + q] >= 0) info[o + q] = -1;
        }
        return;
    }
    const int32_t D = t.D;
    const float lr = a.lr;
    E* __restrict__ S = static_cast<E*>(t.S);
    E* __restrict__ T = static_cast<E*>(t.T);
    float loss = 0.f;

    // Every index of the positive is loaded before any of them is used, so
    // the loads overlap; ids were validated when the batch was grouped and
    // are checked again so that a batch changed before its apply is reported
    // instead of read out of bounds.
    // Batch indices fit in 32 bits (the configuration bounds max_batch (2 + K)
    // below 2^31), so the batch arrays are addressed as a base plus a 32-bit
    // offset.
    bool active = i < a.n;
    int32_t u = 0, v = 0, info_s = -1, info_d = -1;
    float c_i = 0.f;
    int32_t mk[NB], ik[NB];
    const uint32_t i32 = (uint32_t)i;
    const uint32_t o = i32 * (uint32_t)(2 + K);
    const uint32_t nbase = i32 * neg_stride;
    int cnt = K < NB ? K : NB;
    if (active) {
        u = a.src[i32];
        v = a.dst[i32];
        c_i = positive_weight(a, i32);
        info_s = info[o];
        info_d = info[o + 1];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            if (j < cnt) {
                mk[j] = neg[nbase + j];
                ik[j] = info[o + 2 + j];
            }
        }
        if (lane == 0) {
            if (info_s >= 0) info[o] = -1;
            if (info_d >= 0) info[o + 1] = -1;
#pragma unroll
            for (int j = 0; j < NB; ++j)
                if (j < cnt && ik[j] >= 0) info[o + 2 + j] = -1;
        }
        if (u < 0 || (int64_t)u >= t.N || v < 0 || (int64_t)v >= t.N) {
            if (lane == 0) raise_internal(ctl, kSiteStepIds);
            active = false;
        }
    }
    if (active) {
        const float c = c_i;
        float4 s[C], dS[C];
        Reg t0[R];
        Reg tk[NB][R];
        IO::load(s, S, u, D, lane);
        IO::load_packed(t0, T, v, D, lane);
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < cnt) IO::load_packed(tk[j], T, mk[j], D, lane);

        // positive pair
        const float x = group_sum<G>(IO::dotp(s, t0));
        IO::refresh(t0);
        // g: the positive's coefficient; dS: the source row's gradient
        float g = 0.f;
        float lsum = 0.f;
        auto positive_update = [&]() {
#pragma unroll
            for (int q = 0; q < C; ++q) dS[q] = scale4(g, IO::chunk(t0, q));
            if (info_d < 0) {
                float4 nv[C];
#pragma unroll
                for (int q = 0; q < C; ++q) nv[q] = axpy4(-(lr * g), s[q], IO::chunk(t0, q));
                IO::store(T, v, D, lane, nv);
            } else {
                float4 cv[C];
#pragma unroll
                for (int q = 0; q < C; ++q) cv[q] = scale4(g, s[q]);
                DIO::store(dup, info_d, D, lane, cv);
            }
        };
        if constexpr (!kLanePos) {
            g = coef_pos(c, x);
            // with lane coefficients every lane's terms are summed: the
            // positive's term is lane 0's
            if (!kLaneCoefs || lane == 0) lsum = softplus_f(-x);
            positive_update();
        }

        // negatives, NB rows in flight at a time
        int kb = 0;
        while (true) {
            float y[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) y[j] = (j < cnt) ? IO::dotp(s, tk[j]) : 0.f;
#pragma unroll
            for (int j = 0; j < NB; ++j) y[j] = group_sum<G>(y[j]);
#pragma unroll
            for (int j = 0; j < NB; ++j) IO::refresh(tk[j]);
            float h[NB];
            if constexpr (kLaneCoefs) {
                // lane q of the group evaluates value q -- the positive's
                // -x (q = 0, first block only, with kLanePos) or negative
                // q - 1's y -- and the group reads the coefficients from
                // those lanes:
                //   coefficient sign c sigmoid(z), loss term softplus(z),
                // both from e = exp(-|z|) (no overflow)
                float z = lane == 0 ? -x : 0.f;
                bool has = kLanePos && lane == 0 && kb == 0;
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    if (lane == j + 1) {
                        z = y[j];
                        has = j < cnt;
                    }
                }
                const float e = expf(-fabsf(z));
                const float coef = (lane == 0 ? -c : c) * (z >= 0.f ? 1.0f : e) / (1.0f + e);
                if (has) lsum += fmaxf(z, 0.f) + log1pf(e);
                const int first = (int)(threadIdx.x & 63u) - lane;  // the group's first lane
                if (kLanePos && kb == 0) {
                    g = __shfl(coef, first, 64);
                    positive_update();
                }
#pragma unroll
                for (int j = 0; j < NB; ++j) h[j] = __shfl(coef, first + 1 + j, 64);
            } else {
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    if (j < cnt) {
                        h[j] = coef_neg(c, y[j]);
                        lsum += softplus_f(y[j]);
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                if (j < cnt) {
#pragma unroll
                    for (int q = 0; q < C; ++q) dS[q] = axpy4(h[j], IO::chunk(tk[j], q), dS[q]);
                    if (ik[j] < 0) {
                        float4 nv[C];
#pragma unroll
                        for (int q = 0; q < C; ++q)
                            nv[q] = axpy4(-(lr * h[j]), s[q], IO::chunk(tk[j], q));
                        IO::store(T, mk[j], D, lane, nv);
                    } else {
                        float4 cv[C];
#pragma unroll
                        for (int q = 0; q < C; ++q) cv[q] = scale4(h[j], s[q]);
                        DIO::store(dup, ik[j], D, lane, cv);
                    }
                }
            }
            kb += NB;
            if (kb >= K) break;
            cnt = (K - kb) < NB ? (K - kb) : NB;
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                if (j < cnt) {
                    mk[j] = neg[nbase + (uint32_t)(kb + j)];
                    ik[j] = info[o + 2 + (uint32_t)(kb + j)];
                }
            }
            if (lane == 0) {
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    if (j < cnt && ik[j] >= 0) info[o + 2 + (uint32_t)(kb + j)] = -1;
            }
#pragma unroll
            for (int j = 0; j < NB; ++j)
                if (j < cnt) IO::load_packed(tk[j], T, mk[j], D, lane);
        }

        // source row
        if (info_s < 0) {
            float4 nv[C];
#pragma unroll
            for (int q = 0; q < C; ++q) nv[q] = axpy4(-lr, dS[q], s[q]);
            IO::store(S, u, D, lane, nv);
        } else {
            DIO::store(dup, info_s, D, lane, dS);
        }
        // with lane coefficients every lane holds its own loss terms
        if (kLaneCoefs || lane == 0) loss = c * lsum;
    }
    block_loss(loss, lossp);
}

// Lanes per row of the fused step and the probe.
static int step_lanes(const TableArgs& t) {
    return uses_pairs(t.dtype, t.D) ? pair_shape(t.D).G : row_shape(t.D).G;
}

static int64_t fused_step_blocks(const TableArgs& t, int64_t n) {
    const int64_t ppb = kBlock / step_lanes(t);
    return (n + ppb - 1) / ppb;
}

hipError_t launch_fused_step(const TableArgs& t, Control* ctl, const StepArgs& a,
                             const int32_t* neg, uint32_t neg_stride, int32_t* info, float* dup,
                             double* lossp, int64_t* blocks_out, hipEvent_t start,
                             hipEvent_t stop, hipStream_t s) {
    const int64_t blocks = fused_step_blocks(t, a.n);
    *blocks_out = blocks;
    if (blocks == 0) return hipSuccess;
    if (uses_pairs(t.dtype, t.D)) {
        HUGE_PAIR_DISPATCH(pair_shape(t.D), {
            HUGE_NEG_DISPATCH(neg_block(t.K), {
                HUGE_FULL_DISPATCH(t.K == NB_, {
                    hipExtLaunchKernelGGL(
                        (k_fused_step<G_, NB_, F_, PairIO<G_, U_, bf16_t>, PairIO<G_, U_, float>>),
                        dim3((unsigned)blocks), dim3(kBlock), 0, s, start, stop, 0, t, ctl, a,
                        neg, neg_stride, info, dup, lossp);
                });
            });
        });
    } else {
        HUGE_ROW_DISPATCH(row_shape(t.D), {
            HUGE_NEG_DISPATCH(neg_block(t.K), {
                HUGE_ELEM_DISPATCH(t.dtype, {
                    HUGE_FULL_DISPATCH(t.K == NB_, {
                        hipExtLaunchKernelGGL(
                            (k_fused_step<G_, NB_, F_, RowIO<G_, C_, E_>, RowIO<G_, C_>>),
                            dim3((unsigned)blocks), dim3(kBlock), 0, s, start, stop, 0, t, ctl,
                            a, neg, neg_stride, info, dup, lossp);
                    });
                });
            });
        });
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Bandwidth probe: the rows one step over the batch touches -- S[u_i],
// T[v_i] and the K negatives T[m_ik] it would draw -- each read and written
// back unchanged, in the fused kernel's launch shape (one group of G lanes per
// positive, NB negative rows in flight), with no arithmetic besides a
// multiplication by a run-time 1.0f that keeps the compiler from dropping the
// stores (x * 1.0f == x for every x).  Its rate is the practical ceiling of
// the step's random row traffic.
// ---------------------------------------------------------------------------
template <int G, int NB, typename IO>
__global__ __launch_bounds__(kBlock) void k_probe(TableArgs t, Control* __restrict__ ctl,
                                                  const int32_t* __restrict__ src,
                                                  const int32_t* __restrict__ dst, int64_t n,
                                                  uint64_t first_pos, float one) {
    using E = typename IO::Elem;
    constexpr int C = IO::C;
    E* __restrict__ S = static_cast<E*>(t.S);
    E* __restrict__ T = static_cast<E*>(t.T);
    constexpr int PPB = kBlock / G;
    const int lane = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * PPB + threadIdx.x / G;
    if (i >= n) return;  // no barrier below
    const int32_t u = src[i], v = dst[i];
    if (u < 0 || (int64_t)u >= t.N || v < 0 || (int64_t)v >= t.N) {
        if (lane == 0) raise_error(ctl, kBadId);
        return;
    }
    const int K = t.K;
    auto touch = [&](float4 (&x)[C]) {
#pragma unroll
        for (int q = 0; q < C; ++q) x[q] = scale4(one, x[q]);
    };
    float4 s[C], t0[C];
    float4 tk[NB][C];
    int32_t mk[NB];
    for (int kb = 0; kb < K; kb += NB) {
        const int cnt = (K - kb) < NB ? (K - kb) : NB;
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < cnt)
                mk[j] = draw_negative(t.seed, first_pos + (uint64_t)i, (uint32_t)(kb + j),
                                      (uint64_t)t.N, t.thr, t.alias);
        if (kb == 0) {
            IO::load(s, S, u, t.D, lane);
            IO::load(t0, T, v, t.D, lane);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (j < cnt) IO::load(tk[j], T, mk[j], t.D, lane);
        if (kb == 0) {
            touch(s);
            touch(t0);
            IO::store(S, u, t.D, lane, s);
            IO::store(T, v, t.D, lane, t0);
        }
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            if (j < cnt) {
                touch(tk[j]);
                IO::store(T, mk[j], t.D, lane, tk[j]);
            }
        }
    }
}

hipError_t launch_probe(const TableArgs& t, Control* ctl, const int32_t* src, const int32_t* dst,
                        int64_t n, uint64_t first_pos, hipStream_t s) {
    const int64_t blocks = fused_step_blocks(t, n);
    if (blocks == 0) return hipSuccess;
    if (uses_pairs(t.dtype, t.D)) {
        HUGE_PAIR_DISPATCH(pair_shape(t.D), {
            HUGE_NEG_DISPATCH(neg_block(t.K), {
                hipLaunchKernelGGL((k_probe<G_, NB_, PairIO<G_, U_, bf16_t>>),
                                   dim3((unsigned)blocks), dim3(kBlock), 0, s, t, ctl, src, dst,
                                   n, first_pos, 1.0f);
            });
        });
    } else {
        HUGE_ROW_DISPATCH(row_shape(t.D), {
            HUGE_NEG_DISPATCH(neg_block(t.K), {
                HUGE_ELEM_DISPATCH(t.dtype, {
                    hipLaunchKernelGGL((k_probe<G_, NB_, RowIO<G_, C_, E_>>),
                                       dim3((unsigned)blocks), dim3(kBlock), 0, s, t, ctl, src,
                                       dst, n, first_pos, 1.0f);
                });
            });
        });
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Repeated rows.  The contributions of a row, at duplicate-buffer slots
// start .. start + len - 1, are added in that order, in double (a hub row can
// collect tens of thousands of terms), and the row is rounded once to its
// element type: row = round(row - lr * sum) (for bf16 tables through fp32).
// ---------------------------------------------------------------------------
struct double4_ {
    double x, y, z, w;
};

__device__ __forceinline__ void addd(double4_& a, float4 b) {
    a.x += (double)b.x;
    a.y += (double)b.y;
    a.z += (double)b.z;
    a.w += (double)b.w;
}

template <int G, int C>
struct PartIO {
    // rows of D doubles, lane l owns elements 4 (l + c G) .. + 3
    __device__ __forceinline__ static void load(double4_ (&x)[C], const double* __restrict__ base,
                                                int64_t row, int32_t D, int lane) {
        const double4_* p = reinterpret_cast<const double4_*>(base + row * (int64_t)D);
        const int q = D >> 2;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int j = lane + c * G;
            x[c] = (j < q) ? p[j] : double4_{0.0, 0.0, 0.0, 0.0};
        }
    }
    __device__ __forceinline__ static void store(double* __restrict__ base, int64_t row,
                                                 int32_t D, int lane, const double4_ (&x)[C]) {
        double4_* p = reinterpret_cast<double4_*>(base + row * (int64_t)D);
        const int q = D >> 2;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int j = lane + c * G;
            if (j < q) p[j] = x[c];
        }
    }
};

template <int G, int C>
__device__ __forceinline__ void sum_rows(double4_ (&acc)[C], const float* __restrict__ rows,
                                         int64_t start, int64_t len, int32_t D, int lane) {
    using IO = RowIO<G, C>;
#pragma unroll
    for (int q = 0; q < C; ++q) acc[q] = double4_{0.0, 0.0, 0.0, 0.0};
    int64_t r = 0;
    for (; r + 4 <= len; r += 4) {
        float4 b0[C], b1[C], b2[C], b3[C];
        IO::load(b0, rows, start + r, D, lane);
        IO::load(b1, rows, start + r + 1, D, lane);
        IO::load(b2, rows, start + r + 2, D, lane);
        IO::load(b3, rows, start + r + 3, D, lane);
#pragma unroll
        for (int q = 0; q < C; ++q) {
            addd(acc[q], b0[q]);
            addd(acc[q], b1[q]);
            addd(acc[q], b2[q]);
            addd(acc[q], b3[q]);
        }
    }
    for (; r < len; ++r) {
        float4 b[C];
        IO::load(b, rows, start + r, D, lane);
#pragma unroll
        for (int q = 0; q < C; ++q) addd(acc[q], b[q]);
    }
}

// The table and row of a key (N + i: source row i, else context row key).
template <typename E>
__device__ __forceinline__ E* key_row(const TableArgs& t, uint32_t key, int64_t* row) {
    const bool src = (int64_t)key >= t.N;
    *row = src ? (int64_t)key - t.N : (int64_t)key;
    return static_cast<E*>(src ? t.S : t.T);
}

// r -= lr g, in double, rounded once to the table's type by the store.
template <int C>
__device__ __forceinline__ void sgd_row(float4 (&r)[C], const double4_ (&g)[C], float lr) {
    const double l = (double)lr;
#pragma unroll
    for (int q = 0; q < C; ++q) {
        r[q].x = (float)((double)r[q].x - l * g[q].x);
        r[q].y = (float)((double)r[q].y - l * g[q].y);
        r[q].z = (float)((double)r[q].z - l * g[q].z);
        r[q].w = (float)((double)r[q].w - l * g[q].w);
    }
}

template <int G, int C, typename E>
__device__ __forceinline__ void apply_row(const TableArgs& t, uint32_t key,
                                          const double4_ (&g)[C], float lr, int lane) {
    using IO = RowIO<G, C, E>;
    int64_t row;
    E* base = key_row<E>(t, key, &row);
    float4 r[C];
    IO::load(r, base, row, t.D, lane);
    sgd_row<C>(r, g, lr);
    IO::store(base, row, t.D, lane, r);
}

// Partial sums of the groups of a workgroup, combined in group order.
template <int G, int C>
__device__ __forceinline__ void coop_store(double* s_part, int grp, int lane, int32_t D,
                                           const double4_ (&acc)[C]) {
    const int q = D >> 2;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int j = lane + c * G;
        if (j < q) reinterpret_cast<double4_*>(s_part + (size_t)grp * D)[j] = acc[c];
    }
}

template <int G, int C>
__device__ __forceinline__ void coop_total(double4_ (&acc)[C], const double* s_part, int lane,
                                           int32_t D) {
    constexpr int PPB = kBlock / G;
    const int q = D >> 2;
#pragma unroll
    for (int c = 0; c < C; ++c) acc[c] = double4_{0.0, 0.0, 0.0, 0.0};
    for (int g = 0; g < PPB; ++g) {
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int j = lane + c * G;
            if (j < q) {
                const double4_ b = reinterpret_cast<const double4_*>(s_part + (size_t)g * D)[j];
                acc[c].x += b.x;
                acc[c].y += b.y;
                acc[c].z += b.z;
                acc[c].w += b.w;
            }
        }
    }
}

// Cooperative sum of `len` rows starting at row `start` of `rows` (fp32
// contributions or fp64 partials): the PPB groups of the workgroup each sum
// a fixed contiguous part, and group 0 receives the parts' sum in group
// order (the result does not depend on scheduling).  Every thread of the
// workgroup calls it; it synchronises twice.
template <int G, int C, typename Row>
__device__ __forceinline__ void coop_sum(double4_ (&acc)[C], const Row* __restrict__ rows,
                                         int64_t start, uint32_t len, int32_t D, int grp,
                                         int lane, double* s_part) {
    constexpr int PPB = kBlock / G;
    const uint32_t part_len = (len + PPB - 1) / PPB;
    const uint32_t b0 = (uint32_t)grp * part_len;
    const uint32_t b1 = b0 + part_len < len ? b0 + part_len : len;
    const int64_t cnt = b1 > b0 ? (int64_t)(b1 - b0) : 0;
    if constexpr (sizeof(Row) == sizeof(float)) {
        sum_rows<G, C>(acc, rows, start + b0, cnt, D, lane);
    } else {
#pragma unroll
        for (int q = 0; q < C; ++q) acc[q] = double4_{0.0, 0.0, 0.0, 0.0};
        for (int64_t r = 0; r < cnt; ++r) {
            double4_ x[C];
            PartIO<G, C>::load(x, rows, start + b0 + r, D, lane);
#pragma unroll
            for (int q = 0; q < C; ++q) {
                acc[q].x += x[q].x;
                acc[q].y += x[q].y;
                acc[q].z += x[q].z;
                acc[q].w += x[q].w;
            }
        }
    }
    coop_store<G, C>(s_part, grp, lane, D, acc);
    __syncthreads();
    if (grp == 0) coop_total<G, C>(acc, s_part, lane, D);
    __syncthreads();
}

// Fixed-order sum of one double per thread over the workgroup (a tree in
// LDS); every thread receives the sum.  Synchronises.
__device__ __forceinline__ double block_sum_fixed(double v, double* s_red) {
    s_red[threadIdx.x] = v;
    __syncthreads();
#pragma unroll
    for (int w = kBlock / 2; w > 0; w >>= 1) {
        if ((int)threadIdx.x < w) s_red[threadIdx.x] += s_red[threadIdx.x + w];
        __syncthreads();
    }
    const double r = s_red[0];
    __syncthreads();
    return r;
}

// After the fused step, in one launch:
//   loss:   workgroup 0 sums the fused step's per-workgroup partials in a
//           fixed order and takes no records, so the sum runs beside them
//           (no cross-workgroup step: a device-scope fence per workgroup,
//           to pass partial sums between them, measured slower);
//   short runs ({start, len <= kShortRun, key}): one thread group each
//           loads the row with its contributions, sums them in occurrence
//           order and updates the row;
//   pieces ({start, len <= kPiece, key, comb}): the whole workgroup sums
//           them; a whole run (comb = 0) updates its row; a piece of a
//           longer run stores its sum as partial z of its combine record
//           {key, first partial, partials, first slot}, and the workgroup
//           that stores the record's last partial (an arrival counter after
//           a device-scope release by the storing wave; an acquire before
//           the partials are read) adds the partials in piece order and
//           updates the row once.
// The records come in one list per kind, their counts in Control (the
// grouping of the batch appended them).
// Exclusive sum of one value per thread over the workgroup; *total receives
// the sum.  Synchronises; s_tmp (kBlock / 64 words) may be reused after the
// next barrier.
__device__ __forceinline__ uint32_t block_excl_sum(uint32_t v, uint32_t* s_tmp, uint32_t* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
    }
    if (lane == 63) s_tmp[wave] = incl;
    __syncthreads();
    uint32_t add = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kBlock / 64; ++w) {
        const uint32_t x = s_tmp[w];
        if (w < wave) add += x;
        all += x;
    }
    *total = all;
    return add + incl - v;
}

// The bucket of record r: the largest b < bins with prefix[b] <= r.
__device__ __forceinline__ int record_bucket(const uint32_t* prefix, int bins, uint32_t r) {
    int lo = 0, hi = bins - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (prefix[mid] <= r) lo = mid; else hi = mid - 1;
    }
    return lo;
}


template <int G, int C, typename E>
__global__ __launch_bounds__(kBlock) void k_finish(TableArgs t, Control* __restrict__ ctl,
                                                   FinishArgs f) {
    constexpr int PPB = kBlock / G;
    __shared__ double s_part[1024 * C];  // PPB x D doubles: D <= 4 G C
    __shared__ double s_red[kBlock];
    __shared__ uint32_t s_flag;
    if (ctl->step_bad) {
        if (blockIdx.x == 0 && threadIdx.x == 0 && f.loss_out != nullptr)
            *f.loss_out = __builtin_nan("");
        return;
    }
    const int grp = threadIdx.x / G;
    const int lane = threadIdx.x % G;
    const int32_t D = t.D;

    // Workgroup 0 (dispatched first) sums the loss and nothing else: thread t
    // adds partial pairs t, t + kBlock, ... in that order (16-byte loads, 32
    // in flight), then the threads' sums meet in a fixed tree: the same
    // double on every run.
    if (blockIdx.x == 0) {
        if (f.loss_out == nullptr) return;
        const double2* p2 = reinterpret_cast<const double2*>(f.lossp);
        const int64_t n2 = f.loss_blocks / 2;
        double acc = 0.0;
        int64_t j = threadIdx.x;
        for (; j + 31 * kBlock < n2; j += 32 * kBlock) {
            double2 v[32];
#pragma unroll
            for (int q = 0; q < 32; ++q) v[q] = p2[j + q * kBlock];
#pragma unroll
            for (int q = 0; q < 32; ++q) {
                acc += v[q].x;
                acc += v[q].y;
            }
        }
        for (; j < n2; j += kBlock) {
            const double2 v = p2[j];
            acc += v.x;
            acc += v.y;
        }
        if (threadIdx.x == 0 && (f.loss_blocks & 1)) acc += f.lossp[f.loss_blocks - 1];
        acc = block_sum_fixed(acc, s_red);
        if (threadIdx.x == 0) *f.loss_out = acc;
        return;
    }
    // the other workgroups take the records
    if (f.m == 0) return;
    uint32_t ns = ctl->nshort, np = ctl->npiece;
    if (ns > f.caps.shorts || np > f.caps.pieces) {  // cannot happen: the grouping checks
        if (threadIdx.x == 0) raise_internal(ctl, kSiteFinishComb);
        ns = ns < f.caps.shorts ? ns : f.caps.shorts;
        np = np < f.caps.pieces ? np : f.caps.pieces;
    }
    const uint32_t rec_groups = gridDim.x - 1u;
    const uint32_t wg = blockIdx.x - 1u;
    for (uint32_t r = wg * PPB + grp; r < ns; r += rec_groups * PPB) {
        const uint4 rec = f.shorts[r];
        // a record is used only if it lies inside this batch (the grouping
        // writes only such records; the check keeps a broken invariant from
        // reaching memory outside the buffers)
        if (rec.y == 0u || rec.y > kShortRun || (int64_t)rec.x + rec.y > f.m ||
            (int64_t)rec.z >= 2 * t.N) {
            if (lane == 0) raise_internal(ctl, kSiteFinishComb);
            continue;
        }
        // the row's values are loaded with the contributions
        int64_t row;
        E* base = key_row<E>(t, rec.z, &row);
        float4 cur[C];
        RowIO<G, C, E>::load(cur, base, row, D, lane);
        double4_ acc[C];
        sum_rows<G, C>(acc, f.dup, rec.x, rec.y, D, lane);
        sgd_row<C>(cur, acc, f.lr);
        RowIO<G, C, E>::store(base, row, D, lane, cur);
    }
    for (uint32_t r = wg; r < np; r += rec_groups) {
        const uint4 rec = f.pieces[r];  // the same for every thread
        if (rec.y == 0u || rec.y > kPiece || (int64_t)rec.x + rec.y > f.m ||
            (int64_t)rec.z >= 2 * t.N) {  // uniform; cannot happen
            if (threadIdx.x == 0) raise_internal(ctl, kSiteFinishComb);
            continue;
        }
        double4_ acc[C];
        coop_sum<G, C>(acc, f.dup, rec.x, rec.y, D, grp, lane, s_part);
        if (rec.w == 0u) {
            if (grp == 0) apply_row<G, C, E>(t, rec.z, acc, f.lr, lane);
            continue;
        }
        const uint32_t ci = rec.w - 1u;
        const uint4 cb = ci < f.caps.combs ? f.combs[ci] : make_uint4(0u, 0u, 0u, 0u);
        const uint32_t z = (rec.x - cb.w) / kPiece;
        if (ci >= f.caps.combs || z >= cb.z || (uint64_t)cb.y + cb.z > f.caps.parts ||
            (int64_t)cb.x >= 2 * t.N) {
            if (threadIdx.x == 0) raise_internal(ctl, kSiteFinishComb);
            continue;  // uniform
        }
        if (grp == 0) PartIO<G, C>::store(f.part, (int64_t)cb.y + z, D, lane, acc);
        // the partial is wave 0's (a group has at most 64 lanes): wave 0
        // alone releases it before its arrival is counted
        if (threadIdx.x < 64) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            if (threadIdx.x == 0) s_flag = atomicAdd(&f.ccount[ci], 1u) == cb.z - 1u ? 1u : 0u;
        }
        __syncthreads();
        if (s_flag) {  // uniform: the last piece of the row
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            coop_sum<G, C>(acc, static_cast<const double*>(f.part), cb.y, cb.z, D, grp, lane,
                           s_part);
            if (grp == 0) apply_row<G, C, E>(t, cb.x, acc, f.lr, lane);
        }
    }
}

hipError_t launch_finish(const TableArgs& t, Control* ctl, const FinishArgs& f, hipEvent_t stop,
                         hipStream_t s) {
    const RowShape rs = row_shape(t.D);
    // workgroup 0 sums the loss; the other 2047 take the repeated-row records
    // (1024 workgroups measured 1 us slower per step at SBM-100M)
    const int64_t grid = 2048;
    HUGE_ROW_DISPATCH(rs, {
        HUGE_ELEM_DISPATCH(t.dtype, {
            hipExtLaunchKernelGGL((k_finish<G_, C_, E_>), dim3((unsigned)grid), dim3(kBlock), 0, s,
                                  nullptr, stop, 0, t, ctl, f);
        });
    });
    return hipGetLastError();
}

}  // namespace huge
