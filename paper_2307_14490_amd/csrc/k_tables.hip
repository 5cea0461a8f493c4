// Table initialisation, row gather, per-call set-up, negative sampling with
// sort-key emission, and the final loss reduction.
#include <math.h>

#include "common.hpp"
#include "device.hpp"

namespace huge {

// ---------------------------------------------------------------------------
// Initial tables: each thread fills one float4 (one Philox block) of one row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_init(float* __restrict__ S, float* __restrict__ T,
                                                 int64_t N, int32_t D, uint64_t seed,
                                                 float scale) {
    const int64_t q = D >> 2;
    const int64_t per_table = N * q;
    const int64_t total = 2 * per_table;
    const uint32_t klo = (uint32_t)seed, khi = (uint32_t)(seed >> 32);
    for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * kBlock) {
        const int table = e >= per_table ? 1 : 0;
        const int64_t f = e - table * per_table;
        const int64_t row = f / q;
        const uint32_t blk = (uint32_t)(f - row * q);
        const uint4 r = philox4x32_10(
            make_uint4((uint32_t)row, (uint32_t)((uint64_t)row >> 32), blk, 2u + table), klo,
            khi);
        float4 v;
        v.x = (float)((int32_t)(r.x >> 8) - 8388608) * scale;
        v.y = (float)((int32_t)(r.y >> 8) - 8388608) * scale;
        v.z = (float)((int32_t)(r.z >> 8) - 8388608) * scale;
        v.w = (float)((int32_t)(r.w >> 8) - 8388608) * scale;
        float* base = table ? T : S;
        reinterpret_cast<float4*>(base + row * (int64_t)D)[blk] = v;
    }
}

hipError_t launch_init(const TableArgs& t, float half_width, hipStream_t s) {
    const float scale = ldexpf(half_width, -23);  // exact: a power-of-two scaling
    const int64_t total = 2 * t.N * (int64_t)(t.D / 4);
    int64_t blocks = (total + kBlock - 1) / kBlock;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_init, dim3((unsigned)blocks), dim3(kBlock), 0, s, t.S, t.T, t.N, t.D,
                       t.seed, scale);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Row gather: one group of 64 lanes per requested row.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_get_rows(const float* __restrict__ table, int64_t N,
                                                     int32_t D, Control* ctl,
                                                     const int64_t* __restrict__ ids, int64_t n,
                                                     float* __restrict__ out) {
    const int64_t r = (int64_t)blockIdx.x * (kBlock / 64) + threadIdx.x / 64;
    const int lane = threadIdx.x & 63;
    if (r >= n) return;
    const int64_t id = ids[r];
    const int q = D >> 2;
    float4* o = reinterpret_cast<float4*>(out + r * (int64_t)D);
    if (id < 0 || id >= N) {
        if (lane == 0) atomicCAS(&ctl->error, 0u, kBadId);
        const float nan = __builtin_nanf("");
        for (int j = lane; j < q; j += 64) o[j] = make_float4(nan, nan, nan, nan);
        return;
    }
    const float4* p = reinterpret_cast<const float4*>(table + id * (int64_t)D);
    for (int j = lane; j < q; j += 64) o[j] = p[j];
}

hipError_t launch_get_rows(const TableArgs& t, Control* ctl, int32_t table, const int64_t* ids,
                           int64_t n, float* out, hipStream_t s) {
    const int64_t blocks = (n + 3) / 4;
    hipLaunchKernelGGL(k_get_rows, dim3((unsigned)blocks), dim3(kBlock), 0, s,
                       table ? t.T : t.S, t.N, t.D, ctl, ids, n, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per-call set-up: clear the call's flag, the tile tickets, the sort's
// overflow flag and queue count, and the digit histograms (a kernel rather
// than a memset so that the sequence stays valid inside a captured graph).
// ---------------------------------------------------------------------------
__global__ void k_begin(Control* ctl, uint32_t* hist) {
    const int t = threadIdx.x;
    if (hist != nullptr)
        for (int i = t; i < kMaxPasses * kMaxBins; i += blockDim.x) hist[i] = 0u;
    if (t == 0) {
        ctl->step_bad = 0u;
        for (int p = 0; p < kMaxPasses; ++p) ctl->tickets[p] = 0u;
        ctl->overflow = 0u;
        ctl->big_count = 0u;
    }
}

hipError_t launch_begin(Control* ctl, uint32_t* hist, hipStream_t s) {
    hipLaunchKernelGGL(k_begin, dim3(1), dim3(kBlock), 0, s, ctl, hist);
    return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_clear_u64(uint64_t* p, int64_t words) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < words;
         i += (int64_t)gridDim.x * kBlock)
        p[i] = 0ull;
}

__global__ __launch_bounds__(kBlock) void k_fill_i32(int32_t* p, int32_t v, int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kBlock)
        p[i] = v;
}

hipError_t launch_fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s) {
    int64_t blocks = (n + kBlock - 1) / kBlock;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_fill_i32, dim3((unsigned)blocks), dim3(kBlock), 0, s, p, v, n);
    return hipGetLastError();
}

hipError_t launch_clear_status(uint64_t* status, int64_t words, hipStream_t s) {
    int64_t blocks = (words + kBlock - 1) / kBlock;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_clear_u64, dim3((unsigned)blocks), dim3(kBlock), 0, s, status, words);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Validation, negatives and sort keys.  kSamplePer positives per thread
// (coalesced rounds of one workgroup width); for each positive i:
//   - checks 0 <= src, dst < N and co_count >= 0 (a failure flags the call);
//   - draws the K negatives into neg[i K + k];
//   - if keys != nullptr, writes the (2 + K) occurrence keys of positive i at
//     o = i (2 + K) + slot: slot 0 the source row (key N + src), slot 1 the
//     destination row (key dst), slots 2.. the negatives (key m), sets their
//     info entries to -1 (the run marking overwrites repeated ones) and
//     counts the digits of every radix pass (digit ps = bits [ps * bits,
//     (ps + 1) * bits) of the key, counted at hist[ps * kMaxBins + digit]).
// Without src (src == nullptr) only negatives are drawn.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_sample(TableArgs t, Control* ctl, StepArgs a,
                                                   int32_t* __restrict__ neg,
                                                   uint32_t* __restrict__ keys,
                                                   int32_t* __restrict__ info,
                                                   uint32_t* __restrict__ hist, int passes,
                                                   int bits) {
    __shared__ uint32_t s_hist[kMaxPasses * kMaxBins];
    const bool with_keys = keys != nullptr;
    const uint32_t dmask = (1u << bits) - 1u;
    if (with_keys) {
        for (int j = threadIdx.x; j < passes * kMaxBins; j += kBlock) s_hist[j] = 0u;
        __syncthreads();
    }
    const int K = t.K;
    for (int r = 0; r < kSamplePer; ++r) {
        const int64_t i = ((int64_t)blockIdx.x * kSamplePer + r) * kBlock + threadIdx.x;
        if (i >= a.n) break;
        const uint64_t p = a.first_pos + (uint64_t)i;
        uint32_t key_s = 0, key_d = 0;
        if (a.src != nullptr) {
            int32_t u = a.src[i], v = a.dst[i];
            const int32_t c = a.cc[i];
            if (u < 0 || (int64_t)u >= t.N || v < 0 || (int64_t)v >= t.N) {
                raise_error(ctl, kBadId);
                u = 0;
                v = 0;
            }
            if (c < 0) raise_error(ctl, kBadCount);
            key_s = (uint32_t)((uint64_t)t.N + (uint64_t)u);
            key_d = (uint32_t)v;
        }
        const int64_t o = i * (int64_t)(2 + K);
        if (with_keys) {
            keys[o] = key_s;
            keys[o + 1] = key_d;
            for (int sl = 0; sl < 2 + K; ++sl) info[o + sl] = -1;
            for (int ps = 0; ps < passes; ++ps) {
                atomicAdd(&s_hist[ps * kMaxBins + ((key_s >> (ps * bits)) & dmask)], 1u);
                atomicAdd(&s_hist[ps * kMaxBins + ((key_d >> (ps * bits)) & dmask)], 1u);
            }
        }
        // negatives in chunks of kNegBlock: the alias-table loads of a chunk
        // are independent and issued together
        for (int k0 = 0; k0 < K; k0 += kNegBlock) {
            int32_t mm[kNegBlock];
#pragma unroll
            for (int q = 0; q < kNegBlock; ++q)
                if (k0 + q < K)
                    mm[q] = draw_negative(t.seed, p, (uint32_t)(k0 + q), (uint64_t)t.N, t.thr,
                                          t.alias);
#pragma unroll
            for (int q = 0; q < kNegBlock; ++q) {
                if (k0 + q < K) {
                    const int32_t m = mm[q];
                    neg[i * K + k0 + q] = m;
                    if (with_keys) {
                        keys[o + 2 + k0 + q] = (uint32_t)m;
                        for (int ps = 0; ps < passes; ++ps)
                            atomicAdd(&s_hist[ps * kMaxBins + (((uint32_t)m >> (ps * bits)) & dmask)],
                                      1u);
                    }
                }
            }
        }
    }
    if (with_keys) {
        __syncthreads();
        for (int j = threadIdx.x; j < passes * kMaxBins; j += kBlock) {
            const uint32_t c = s_hist[j];
            if (c) atomicAdd(&hist[j], c);
        }
    }
}

hipError_t launch_sample(const TableArgs& t, Control* ctl, const StepArgs& a, int32_t* neg,
                         uint32_t* keys, int32_t* info, uint32_t* hist, SortPlan plan,
                         hipStream_t s) {
    const int64_t per_block = (int64_t)kBlock * kSamplePer;
    const int64_t blocks = (a.n + per_block - 1) / per_block;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_sample, dim3((unsigned)blocks), dim3(kBlock), 0, s, t, ctl, a, neg, keys,
                       info, hist, keys ? plan.passes : 0, plan.bits);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Loss: fixed-order sum of the per-workgroup partials in double.  A flagged
// call reports NaN.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_loss_final(const Control* ctl,
                                                       const double* __restrict__ part,
                                                       int64_t nb, double* out) {
    __shared__ double s[kBlock];
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < nb; j += kBlock) acc += part[j];
    s[threadIdx.x] = acc;
    __syncthreads();
    for (int w = kBlock / 2; w > 0; w >>= 1) {
        if (threadIdx.x < w) s[threadIdx.x] += s[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = ctl->step_bad ? __builtin_nan("") : s[0];
}

hipError_t launch_loss_final(Control* ctl, const double* lossp, int64_t blocks, double* out,
                             hipStream_t s) {
    hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(kBlock), 0, s, ctl, lossp, blocks, out);
    return hipGetLastError();
}

}  // namespace huge
