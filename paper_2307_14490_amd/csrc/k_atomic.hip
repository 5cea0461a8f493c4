// The atomicAdd variant of the step, and the forward-only loss evaluation.
//
// Atomic variant: three kernels keep the step synchronous without grouping
// rows.  (a) gathers every row and computes the coefficients and the source
// gradient; (b) adds -lr coef S[u] into the context rows with fp32 atomics
// (S still holds pre-step values); (c) adds -lr dS into the source rows.
// The result equals the sorted variant's up to the order of the additions.
// It works on float tables only (bf16 has no native atomic add of the
// precision the step needs); the loss evaluation reads either element type.
#include "common.hpp"
#include "device.hpp"
#include "dispatch.hpp"

namespace huge {

__device__ __forceinline__ void block_loss_a(float loss, double* __restrict__ out) {
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

// Forward for one positive: fills the loss sum and, when coef != nullptr,
// the (1 + K) coefficients and the source gradient.
template <int G, int C, bool kDrawInline, typename E>
__device__ __forceinline__ float forward_positive(const TableArgs& t, const StepArgs& a, int64_t i,
                                                  int32_t u, int32_t v, float c,
                                                  const int32_t* __restrict__ neg, int lane,
                                                  float* __restrict__ coef,
                                                  float* __restrict__ gsrc) {
    using IO = RowIO<G, C, E>;
    const E* __restrict__ S = static_cast<const E*>(t.S);
    const E* __restrict__ T = static_cast<const E*>(t.T);
    const int K = t.K;
    const int32_t D = t.D;
    float4 s[C], t0[C], dS[C];
    IO::load(s, S, u, D, lane);
    IO::load(t0, T, v, D, lane);
    const float x = group_sum<G>(IO::dot(s, t0));
    const float g = coef_pos(c, x);
    float lsum = softplus_f(-x);
    if (coef) {
        if (lane == 0) coef[i * (int64_t)(1 + K)] = g;
#pragma unroll
        for (int q = 0; q < C; ++q) dS[q] = scale4(g, t0[q]);
    }
    for (int kb = 0; kb < K; kb += kNegBlock) {
        const int cnt = (K - kb) < kNegBlock ? (K - kb) : kNegBlock;
        float4 tk[kNegBlock][C];
        int32_t mk[kNegBlock];
#pragma unroll
        for (int j = 0; j < kNegBlock; ++j) {
            if (j < cnt) {
                if (kDrawInline)
                    mk[j] = draw_negative(t.seed, a.first_pos + (uint64_t)i, (uint32_t)(kb + j),
                                          (uint64_t)t.N, t.thr, t.alias);
                else
                    mk[j] = neg[i * (int64_t)K + kb + j];
            }
        }
#pragma unroll
        for (int j = 0; j < kNegBlock; ++j)
            if (j < cnt) IO::load(tk[j], T, mk[j], D, lane);
        float y[kNegBlock];
#pragma unroll
        for (int j = 0; j < kNegBlock; ++j) y[j] = (j < cnt) ? IO::dot(s, tk[j]) : 0.f;
#pragma unroll
        for (int j = 0; j < kNegBlock; ++j) y[j] = group_sum<G>(y[j]);
#pragma unroll
        for (int j = 0; j < kNegBlock; ++j) {
            if (j < cnt) {
                lsum += softplus_f(y[j]);
                if (coef) {
                    const float h = coef_neg(c, y[j]);
                    if (lane == 0) coef[i * (int64_t)(1 + K) + 1 + kb + j] = h;
#pragma unroll
                    for (int q = 0; q < C; ++q) dS[q] = axpy4(h, tk[j][q], dS[q]);
                }
            }
        }
    }
    if (coef) RowIO<G, C>::store(gsrc, i, D, lane, dS);
    return c * lsum;
}

template <int G, int C>
__global__ __launch_bounds__(kBlock) void k_atomic_gather(TableArgs t, Control* __restrict__ ctl,
                                                          StepArgs a,
                                                          const int32_t* __restrict__ neg,
                                                          float* __restrict__ gsrc,
                                                          float* __restrict__ coef,
                                                          double* __restrict__ lossp) {
    if (ctl->step_bad) return;
    constexpr int PPB = kBlock / G;
    const int lane = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * PPB + threadIdx.x / G;
    float loss = 0.f;
    if (i < a.n) {
        // validated when the batch was grouped; checked again so that a batch
        // changed before its apply is reported instead of read out of bounds
        const int32_t u = a.src[i], v = a.dst[i];
        if (u >= 0 && (int64_t)u < t.N && v >= 0 && (int64_t)v < t.N) {
            const float l = forward_positive<G, C, false, float>(
                t, a, i, u, v, positive_weight(a, i), neg, lane, coef, gsrc);
            if (lane == 0) loss = l;
        } else if (lane == 0) {
            raise_internal(ctl, kSiteAtomicIds);
        }
    }
    block_loss_a(loss, lossp);
}

template <int G, int C>
__global__ __launch_bounds__(kBlock) void k_atomic_scatter_T(TableArgs t,
                                                             const Control* __restrict__ ctl,
                                                             StepArgs a,
                                                             const int32_t* __restrict__ neg,
                                                             const float* __restrict__ coef) {
    using IO = RowIO<G, C>;
    if (ctl->step_bad) return;
    constexpr int PPB = kBlock / G;
    const int lane = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * PPB + threadIdx.x / G;
    if (i >= a.n) return;
    const int32_t u = a.src[i], v = a.dst[i];
    if (u < 0 || (int64_t)u >= t.N || v < 0 || (int64_t)v >= t.N) return;
    const int K = t.K;
    const int32_t D = t.D;
    const int q4 = D >> 2;
    float4 s[C];
    IO::load(s, static_cast<const float*>(t.S), u, D, lane);
    for (int j = 0; j <= K; ++j) {
        const int64_t row = j == 0 ? (int64_t)v : (int64_t)neg[i * (int64_t)K + j - 1];
        const float w = -a.lr * coef[i * (int64_t)(1 + K) + j];
        float* p = static_cast<float*>(t.T) + row * (int64_t)D;
#pragma unroll
        for (int q = 0; q < C; ++q) {
            const int jj = lane + q * G;
            if (jj < q4) {
                unsafeAtomicAdd(p + 4 * jj + 0, w * s[q].x);
                unsafeAtomicAdd(p + 4 * jj + 1, w * s[q].y);
                unsafeAtomicAdd(p + 4 * jj + 2, w * s[q].z);
                unsafeAtomicAdd(p + 4 * jj + 3, w * s[q].w);
            }
        }
    }
}

template <int G, int C>
__global__ __launch_bounds__(kBlock) void k_atomic_scatter_S(TableArgs t,
                                                             const Control* __restrict__ ctl,
                                                             StepArgs a,
                                                             const float* __restrict__ gsrc) {
    using IO = RowIO<G, C>;
    if (ctl->step_bad) return;
    constexpr int PPB = kBlock / G;
    const int lane = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * PPB + threadIdx.x / G;
    if (i >= a.n) return;
    const int32_t u = a.src[i];
    if (u < 0 || (int64_t)u >= t.N) return;
    const int32_t D = t.D;
    const int q4 = D >> 2;
    float4 g[C];
    IO::load(g, gsrc, i, D, lane);
    float* p = static_cast<float*>(t.S) + (int64_t)u * D;
    const float w = -a.lr;
#pragma unroll
    for (int q = 0; q < C; ++q) {
        const int jj = lane + q * G;
        if (jj < q4) {
            unsafeAtomicAdd(p + 4 * jj + 0, w * g[q].x);
            unsafeAtomicAdd(p + 4 * jj + 1, w * g[q].y);
            unsafeAtomicAdd(p + 4 * jj + 2, w * g[q].z);
            unsafeAtomicAdd(p + 4 * jj + 3, w * g[q].w);
        }
    }
}

// Loss of a batch at the current tables; validates ids and counts itself and
// draws the negatives inline (no workspace for them).
template <int G, int C, typename E>
__global__ __launch_bounds__(kBlock) void k_eval(TableArgs t, Control* __restrict__ ctl, StepArgs a,
                                                 double* __restrict__ lossp) {
    constexpr int PPB = kBlock / G;
    const int lane = threadIdx.x % G;
    const int64_t i = (int64_t)blockIdx.x * PPB + threadIdx.x / G;
    float loss = 0.f;
    if (i < a.n) {
        const int32_t u = a.src[i], v = a.dst[i];
        const bool ok_id = u >= 0 && (int64_t)u < t.N && v >= 0 && (int64_t)v < t.N;
        const float c = weight_valid(a, i) ? positive_weight(a, i) : -1.f;
        if (!ok_id || c < 0.f) {
            if (lane == 0) raise_error(ctl, ok_id ? kBadCount : kBadId);
        } else {
            const float l = forward_positive<G, C, true, E>(t, a, i, u, v, c, nullptr, lane,
                                                            nullptr, nullptr);
            if (lane == 0) loss = l;
        }
    }
    block_loss_a(loss, lossp);
}

static int64_t blocks_for(int dim, int64_t n) {
    const RowShape rs = row_shape(dim);
    const int64_t ppb = kBlock / rs.G;
    return (n + ppb - 1) / ppb;
}

hipError_t launch_atomic_gather(const TableArgs& t, Control* ctl, const StepArgs& a,
                                const int32_t* neg, float* gsrc, float* coef, double* lossp,
                                int64_t* blocks_out, hipStream_t s) {
    const RowShape rs = row_shape(t.D);
    const int64_t blocks = blocks_for(t.D, a.n);
    *blocks_out = blocks;
    if (blocks == 0) return hipSuccess;
    HUGE_ROW_DISPATCH(rs, {
        hipLaunchKernelGGL((k_atomic_gather<G_, C_>), dim3((unsigned)blocks), dim3(kBlock), 0, s,
                           t, ctl, a, neg, gsrc, coef, lossp);
    });
    return hipGetLastError();
}

hipError_t launch_atomic_scatter_T(const TableArgs& t, Control* ctl, const StepArgs& a,
                                   const int32_t* neg, const float* coef, hipStream_t s) {
    const RowShape rs = row_shape(t.D);
    const int64_t blocks = blocks_for(t.D, a.n);
    if (blocks == 0) return hipSuccess;
    HUGE_ROW_DISPATCH(rs, {
        hipLaunchKernelGGL((k_atomic_scatter_T<G_, C_>), dim3((unsigned)blocks), dim3(kBlock), 0,
                           s, t, ctl, a, neg, coef);
    });
    return hipGetLastError();
}

hipError_t launch_atomic_scatter_S(const TableArgs& t, Control* ctl, const StepArgs& a,
                                   const float* gsrc, hipStream_t s) {
    const RowShape rs = row_shape(t.D);
    const int64_t blocks = blocks_for(t.D, a.n);
    if (blocks == 0) return hipSuccess;
    HUGE_ROW_DISPATCH(rs, {
        hipLaunchKernelGGL((k_atomic_scatter_S<G_, C_>), dim3((unsigned)blocks), dim3(kBlock), 0,
                           s, t, ctl, a, gsrc);
    });
    return hipGetLastError();
}

hipError_t launch_eval(const TableArgs& t, Control* ctl, const StepArgs& a, double* lossp,
                       int64_t* blocks_out, hipStream_t s) {
    const RowShape rs = row_shape(t.D);
    const int64_t blocks = blocks_for(t.D, a.n);
    *blocks_out = blocks;
    if (blocks == 0) return hipSuccess;
    HUGE_ROW_DISPATCH(rs, {
        HUGE_ELEM_DISPATCH(t.dtype, {
            hipLaunchKernelGGL((k_eval<G_, C_, E_>), dim3((unsigned)blocks), dim3(kBlock), 0, s,
                               t, ctl, a, lossp);
        });
    });
    return hipGetLastError();
}

}  // namespace huge
