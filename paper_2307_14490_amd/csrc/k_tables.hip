// Table initialisation, row gather, per-call set-up, negative sampling with
// sort-key emission, and the final loss reduction.
#include <math.h>

#include "common.hpp"
#include "device.hpp"
#include "dispatch.hpp"

namespace huge {

// ---------------------------------------------------------------------------
// Initial tables: each thread fills one chunk of four elements (one Philox
// block) of one row.  The values are exact in float; a bf16 table holds them
// rounded to nearest, ties to even.
// ---------------------------------------------------------------------------
template <typename E>
__global__ __launch_bounds__(kBlock) void k_init(E* __restrict__ S, E* __restrict__ T,
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
        E* base = table ? T : S;
        store_chunk(base + row * (int64_t)D, (int)blk, v);
    }
}

hipError_t launch_init(const TableArgs& t, float half_width, hipStream_t s) {
    const float scale = ldexpf(half_width, -23);  // exact: a power-of-two scaling
    const int64_t total = 2 * t.N * (int64_t)(t.D / 4);
    int64_t blocks = (total + kBlock - 1) / kBlock;
    if (blocks > 65536) blocks = 65536;
    HUGE_ELEM_DISPATCH(t.dtype, {
        hipLaunchKernelGGL(k_init<E_>, dim3((unsigned)blocks), dim3(kBlock), 0, s,
                           static_cast<E_*>(t.S), static_cast<E_*>(t.T), t.N, t.D, t.seed, scale);
    });
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Row gather: one group of 64 lanes per requested row; rows of a bf16 table
// are widened to float (exactly).
// ---------------------------------------------------------------------------
template <typename E>
__global__ __launch_bounds__(kBlock) void k_get_rows(const E* __restrict__ table, int64_t N,
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
    const E* p = table + id * (int64_t)D;
    for (int j = lane; j < q; j += 64) o[j] = load_chunk(p, j);
}

hipError_t launch_get_rows(const TableArgs& t, Control* ctl, int32_t table, const int64_t* ids,
                           int64_t n, float* out, hipStream_t s) {
    const int64_t blocks = (n + 3) / 4;
    HUGE_ELEM_DISPATCH(t.dtype, {
        hipLaunchKernelGGL(k_get_rows<E_>, dim3((unsigned)blocks), dim3(kBlock), 0, s,
                           static_cast<const E_*>(table ? t.T : t.S), t.N, t.D, ctl, ids, n, out);
    });
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per-call set-up: clear the call's flag (a kernel rather than a memset so
// that the sequence stays valid inside a captured graph).
// ---------------------------------------------------------------------------
__global__ HUGE_BESIDE void k_begin(Control* ctl) {
    if (threadIdx.x == 0) {
        ctl->step_bad = 0u;
        ctl->nshort = 0u;
        ctl->npiece = 0u;
    }
}

hipError_t launch_begin(Control* ctl, hipStream_t s) {
    hipLaunchKernelGGL(k_begin, dim3(1), dim3(64), 0, s, ctl);
    return hipGetLastError();
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


// ---------------------------------------------------------------------------
// Validation, negatives and sort keys.  A workgroup takes P consecutive
// positives (P = sample_tile_positives(K, n) with keys, else kSamplePos).
// Positive i has S = 2 + K occurrences at o = i S + slot: slot 0 the source
// row (key N + src), slot 1 the destination row (key dst), slot 2 + k
// negative k (key m).
//   - one thread per positive checks 0 <= src, dst < N and co_count >= 0 (a
//     failure flags the call) and, with keys, writes keys of slots 0 and 1;
//   - one thread per negative, consecutive threads on consecutive (i, k), so
//     that the stores of a wave are contiguous, draws negative k of positive
//     i into neg[i K + k] (if neg is not null) and, with keys, keys[o] of
//     slot 2 + k.
// With keys, the workgroup's P S keys are one tile of the radix pass: their
// counts per digit (lowest `bits` bits) go to LDS as they are written and
// then to tcount[workgroup * 2^bits + digit].
// Without src only negatives are drawn.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) HUGE_BESIDE void k_sample(TableArgs t, Control* ctl,
                                                               StepArgs a,
                                                               int32_t* __restrict__ neg,
                                                               uint32_t* __restrict__ keys,
                                                               uint32_t* __restrict__ tcount,
                                                               int bits, int64_t per_wg) {
    __shared__ uint32_t s_cnt[kMaxBins];
    const bool with_keys = keys != nullptr;
    const uint32_t dmask = (1u << bits) - 1u;
    if (with_keys) {
        for (int d = threadIdx.x; d < (1 << bits); d += kBlock) s_cnt[d] = 0u;
        __syncthreads();
    }
    const int64_t K = t.K, S = 2 + K;
    const int64_t i0 = (int64_t)blockIdx.x * per_wg;
    const int64_t np = a.n - i0 < per_wg ? a.n - i0 : per_wg;  // positives here
    if (a.src != nullptr) {
        for (int64_t j = threadIdx.x; j < np; j += kBlock) {
            const int64_t i = i0 + j;
            int32_t u = a.src[i], v = a.dst[i];
            if (u < 0 || (int64_t)u >= t.N || v < 0 || (int64_t)v >= t.N) {
                raise_error(ctl, kBadId);
                u = 0;
                v = 0;
            }
            if (!weight_valid(a, i)) raise_error(ctl, kBadCount);
            if (with_keys) {
                const uint32_t ks = (uint32_t)((uint64_t)t.N + (uint64_t)u);
                keys[i * S] = ks;
                keys[i * S + 1] = (uint32_t)v;
                atomicAdd(&s_cnt[ks & dmask], 1u);
                atomicAdd(&s_cnt[(uint32_t)v & dmask], 1u);
            }
        }
    }
    // negatives: draw j of this workgroup is negative k of positive i0 + q,
    // j = q K + k; a round of kBlock draws advances (q, k) by dq K + dr
    const uint32_t Ku = (uint32_t)K;
    const uint32_t nd = (uint32_t)(np * K);
    const uint32_t dq = (uint32_t)kBlock / Ku, dr = (uint32_t)kBlock - dq * Ku;
    uint32_t q = (uint32_t)threadIdx.x / Ku, k = (uint32_t)threadIdx.x - q * Ku;
    for (uint32_t j = threadIdx.x; j < nd; j += kBlock) {
        const int64_t i = i0 + q;
        const int32_t m = draw_negative(t.seed, a.first_pos + (uint64_t)i, k, (uint64_t)t.N,
                                        t.thr, t.alias);
        if (neg != nullptr) neg[i * K + k] = m;
        if (with_keys) {
            keys[i * S + 2 + k] = (uint32_t)m;
            atomicAdd(&s_cnt[(uint32_t)m & dmask], 1u);
        }
        k += dr;
        q += dq;
        if (k >= Ku) {
            k -= Ku;
            ++q;
        }
    }
    if (with_keys) {
        __syncthreads();
        for (int d = threadIdx.x; d < (1 << bits); d += kBlock)
            tcount[(int64_t)blockIdx.x * (1 << bits) + d] = s_cnt[d];
    }
}

hipError_t launch_sample(const TableArgs& t, Control* ctl, const StepArgs& a, int32_t* neg,
                         uint32_t* keys, uint32_t* tcount, int bits, hipStream_t s) {
    if (t.K < 1 || t.K > kBlock) return hipErrorInvalidValue;
    if (keys != nullptr && (tcount == nullptr || bits < kMinDigitBits || bits > kMaxDigitBits))
        return hipErrorInvalidValue;
    const int64_t per_wg = keys != nullptr ? sample_tile_positives(t.K, a.n) : kSamplePos;
    if (per_wg < 1) return hipErrorInvalidValue;
    const int64_t blocks = (a.n + per_wg - 1) / per_wg;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_sample, dim3((unsigned)blocks), dim3(kBlock), 0, s, t, ctl, a, neg, keys,
                       tcount, keys != nullptr ? bits : kMinDigitBits, per_wg);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Weights from distance histograms: w_i = sum_d wd[d] hist[i window + d],
// products and sums in double rounded once each (no fused multiply-add), d
// ascending, then rounded once to float.  A negative count gives NaN.
// ---------------------------------------------------------------------------
struct DistWeights {
    float w[kMaxHistWindow];
};

__global__ __launch_bounds__(kBlock) void k_cocount_weights(const int32_t* __restrict__ hist,
                                                            int64_t n, int window, DistWeights wd,
                                                            float* __restrict__ out) {
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    double sum = 0.0;
    bool bad = false;
    for (int d = 0; d < window; ++d) {
        const int32_t h = hist[i * window + d];
        bad = bad || h < 0;
        sum = __dadd_rn(sum, __dmul_rn((double)wd.w[d], (double)h));
    }
    out[i] = bad ? __builtin_nanf("") : __double2float_rn(sum);
}

hipError_t launch_cocount_weights(const int32_t* hist, int64_t n, int window, const float* wd,
                                  float* out, hipStream_t s) {
    if (n == 0) return hipSuccess;
    if (window < 1 || window > kMaxHistWindow) return hipErrorInvalidValue;
    DistWeights W;
    for (int d = 0; d < kMaxHistWindow; ++d) W.w[d] = d < window ? wd[d] : 0.f;
    hipLaunchKernelGGL(k_cocount_weights, dim3((unsigned)((n + kBlock - 1) / kBlock)),
                       dim3(kBlock), 0, s, hist, n, window, W, out);
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
