// Device helpers: counter-based random numbers, negative draws, row access in
// groups of lanes, and the loss pieces.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"

namespace huge {

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of the 4x32
// multiply-xor bijection; the key advances by the Weyl constants between
// rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 ctr, uint32_t key_lo, uint32_t key_hi) {
    constexpr uint32_t kMulA = 0xD2511F53u;
    constexpr uint32_t kMulB = 0xCD9E8D57u;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint32_t ha = __umulhi(kMulA, ctr.x);
        const uint32_t la = kMulA * ctr.x;
        const uint32_t hb = __umulhi(kMulB, ctr.z);
        const uint32_t lb = kMulB * ctr.z;
        ctr = make_uint4(hb ^ ctr.y ^ key_lo, lb, ha ^ ctr.w ^ key_hi, la);
        key_lo += 0x9E3779B9u;
        key_hi += 0xBB67AE85u;
    }
    return ctr;
}

// Negative k of the positive with global index p: a uniform bucket
// floor(x N / 2^64) from the 64-bit word x = (r1 << 32) | r0, then, with an
// alias table, the 32-bit coin r2 keeps the bucket or takes its alias.
__device__ __forceinline__ int32_t draw_negative(uint64_t seed, uint64_t p, uint32_t k,
                                                 uint64_t N, const uint32_t* __restrict__ thr,
                                                 const int32_t* __restrict__ alias) {
    const uint4 r = philox4x32_10(make_uint4((uint32_t)p, (uint32_t)(p >> 32), k, 1u),
                                  (uint32_t)seed, (uint32_t)(seed >> 32));
    const uint64_t x = ((uint64_t)r.y << 32) | (uint64_t)r.x;
    uint64_t j = __umul64hi(x, N);
    if (thr != nullptr) {
        // both table words are loaded before either is used (independent
        // loads); an alias entry outside [0, N) (caller data) keeps j
        const uint32_t th = thr[j];
        const uint64_t a = (uint64_t)(uint32_t)alias[j];
        if (r.z >= th && a < N) j = a;
    }
    return (int32_t)j;
}

// v plus the value of lane (lane XOR OFF), for a v that is already uniform
// over aligned runs of OFF lanes (as it is when the steps of a sum are taken
// in increasing OFF).  Below 16 the partner is read by DPP inside a 16-lane
// row: swap of lane pairs, swap of pairs of pairs, then -- on such v -- the
// mirror inside 8 lanes and inside 16 lanes, which read the partner run's
// value.  At 16 and 32, gfx950's row swaps (v_permlane16_swap: odd rows of
// one copy with even rows of the other; v_permlane32_swap: the two halves)
// give every lane its own and its partner's value.  Both partners form the
// same sum (a + b == b + a), so the result is uniform over 2 OFF lanes.  No
// step goes through LDS.
template <int OFF>
__device__ __forceinline__ float xor_add(float v) {
    const int x = __float_as_int(v);
    if constexpr (OFF == 1) {
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false));
    } else if constexpr (OFF == 2) {
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false));
    } else if constexpr (OFF == 4) {
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false));
    } else if constexpr (OFF == 8) {
        return v + __int_as_float(__builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false));
    } else if constexpr (OFF == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        return __int_as_float(r[0]) + __int_as_float(r[1]);
    } else {
        static_assert(OFF == 32, "a power of two below 64");
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return __int_as_float(r[0]) + __int_as_float(r[1]);
    }
}

// Sum over the G lanes of a group (G a power of two <= 64, groups aligned),
// the same value in every lane of the group; every lane of the group is
// active.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr (G >= 2) v = xor_add<1>(v);
    if constexpr (G >= 4) v = xor_add<2>(v);
    if constexpr (G >= 8) v = xor_add<4>(v);
    if constexpr (G >= 16) v = xor_add<8>(v);
    if constexpr (G >= 32) v = xor_add<16>(v);
    if constexpr (G >= 64) v = xor_add<32>(v);
    return v;
}

// softplus(z) = log(1 + e^z), evaluated without overflow.
__device__ __forceinline__ float softplus_f(float z) {
    return fmaxf(z, 0.0f) + log1pf(expf(-fabsf(z)));
}

// c (sigmoid(x) - 1) = -c / (1 + e^x) and c sigmoid(y) = c / (1 + e^-y).
__device__ __forceinline__ float coef_pos(float c, float x) { return -c / (1.0f + expf(x)); }
__device__ __forceinline__ float coef_neg(float c, float y) { return c / (1.0f + expf(-y)); }

__device__ __forceinline__ float dot4(float4 a, float4 b) {
    return a.x * b.x + a.y * b.y + a.z * b.z + a.w * b.w;
}

__device__ __forceinline__ float4 axpy4(float a, float4 x, float4 y) {
    return make_float4(fmaf(a, x.x, y.x), fmaf(a, x.y, y.y), fmaf(a, x.z, y.z),
                       fmaf(a, x.w, y.w));
}

__device__ __forceinline__ float4 scale4(float a, float4 x) {
    return make_float4(a * x.x, a * x.y, a * x.z, a * x.w);
}

__device__ __forceinline__ float4 add4(float4 a, float4 b) {
    return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
}

__device__ __forceinline__ float4 zero4() { return make_float4(0.f, 0.f, 0.f, 0.f); }

// bfloat16 <-> float.  Widening is exact.  Narrowing rounds to nearest, ties
// to even, on the bit pattern: adding 0x7FFF plus the lowest kept bit carries
// into the kept half exactly when the dropped half is above one half, or
// equal to it with the kept half odd; overflow reaches infinity.  A NaN stays
// a (quiet) NaN.
__device__ __forceinline__ float4 bf16x4_to_float4(uint2 w) {
    return make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xFFFF0000u),
                       __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xFFFF0000u));
}

__device__ __forceinline__ uint32_t float_to_bf16_bits(float f) {
    const uint32_t b = __float_as_uint(f);
    if ((b & 0x7FFFFFFFu) > 0x7F800000u) return (b >> 16) | 0x0040u;
    return (b + 0x7FFFu + ((b >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint2 float4_to_bf16x4(float4 v) {
    return make_uint2(float_to_bf16_bits(v.x) | (float_to_bf16_bits(v.y) << 16),
                      float_to_bf16_bits(v.z) | (float_to_bf16_bits(v.w) << 16));
}

// Chunk j (elements 4j .. 4j + 3) of a row, as float4, for either element type.
__device__ __forceinline__ float4 load_chunk(const float* __restrict__ row, int j) {
    return reinterpret_cast<const float4*>(row)[j];
}
__device__ __forceinline__ float4 load_chunk(const bf16_t* __restrict__ row, int j) {
    return bf16x4_to_float4(reinterpret_cast<const uint2*>(row)[j]);
}
__device__ __forceinline__ void store_chunk(float* __restrict__ row, int j, float4 v) {
    reinterpret_cast<float4*>(row)[j] = v;
}
__device__ __forceinline__ void store_chunk(bf16_t* __restrict__ row, int j, float4 v) {
    reinterpret_cast<uint2*>(row)[j] = float4_to_bf16x4(v);
}

// Four consecutive elements as a kernel keeps them in registers: a float4
// for float tables, the packed uint2 for bf16 tables (widened when used).
template <typename E>
struct Packed4;
template <>
struct Packed4<float> {
    using T = float4;
    __device__ __forceinline__ static T load(const float* __restrict__ row, int j) {
        return reinterpret_cast<const float4*>(row)[j];
    }
    __device__ __forceinline__ static float4 widen(T r) { return r; }
    __device__ __forceinline__ static T zero() { return zero4(); }
    __device__ __forceinline__ static void refresh(T&) {}
};
template <>
struct Packed4<bf16_t> {
    using T = uint2;
    __device__ __forceinline__ static T load(const bf16_t* __restrict__ row, int j) {
        return reinterpret_cast<const uint2*>(row)[j];
    }
    __device__ __forceinline__ static float4 widen(T r) { return bf16x4_to_float4(r); }
    __device__ __forceinline__ static T zero() { return make_uint2(0u, 0u); }
    // an empty asm statement that the compiler must assume redefines r
    __device__ __forceinline__ static void refresh(T& r) { asm volatile("" : "+v"(r.x), "+v"(r.y)); }
};

// Row access policies.  A policy spreads a row of D elements over the G lanes
// of a group as C float4 chunks per lane (chunks past the row read as zero
// and are not stored), and gives the row in two register forms: widened
// (float4[C]) and packed (Reg[R], widened chunk by chunk with chunk()).
// refresh() marks packed registers as redefined, so that chunks used again
// later are widened again from them instead of the widened copies staying
// live in between: widening costs a shift or a mask, registers cost
// occupancy, which hides the latency of the random row accesses.
//
// RowIO: lane l owns the 4-element chunks l, l + G, ..., l + (C-1) G.
template <int G, int CC, typename E = float>
struct RowIO {
    static constexpr int C = CC;
    using Elem = E;
    using P = Packed4<E>;
    using Reg = typename P::T;
    static constexpr int R = CC;
    __device__ __forceinline__ static void load_packed(Reg (&r)[R], const E* __restrict__ base,
                                                       int64_t row, int32_t D, int lane) {
        const E* p = base + row * (int64_t)D;
        const int q = D >> 2;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int j = lane + c * G;
            r[c] = (j < q) ? P::load(p, j) : P::zero();
        }
    }
    __device__ __forceinline__ static float4 chunk(const Reg (&r)[R], int c) {
        return P::widen(r[c]);
    }
    __device__ __forceinline__ static void refresh(Reg (&r)[R]) {
#pragma unroll
        for (int c = 0; c < R; ++c) P::refresh(r[c]);
    }
    __device__ __forceinline__ static void load(float4 (&x)[C], const E* __restrict__ base,
                                                int64_t row, int32_t D, int lane) {
        const E* p = base + row * (int64_t)D;
        const int q = D >> 2;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int j = lane + c * G;
            x[c] = (j < q) ? load_chunk(p, j) : zero4();
        }
    }
    __device__ __forceinline__ static void store(E* __restrict__ base, int64_t row, int32_t D,
                                                 int lane, const float4 (&x)[C]) {
        E* p = base + row * (int64_t)D;
        const int q = D >> 2;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int j = lane + c * G;
            if (j < q) store_chunk(p, j, x[c]);
        }
    }
    __device__ __forceinline__ static float dot(const float4 (&a)[C], const float4 (&b)[C]) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < C; ++c) s += dot4(a[c], b[c]);
        return s;
    }
    __device__ __forceinline__ static float dotp(const float4 (&a)[C], const Reg (&b)[R]) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < C; ++c) s += dot4(a[c], chunk(b, c));
        return s;
    }
};

// PairIO: rows of a multiple of 8 elements in units of 8 (16 bytes of bf16):
// lane l owns the units l, l + G, ..., l + (U-1) G, unit u being the chunks
// 2u and 2u + 1.  With bf16 rows one 16-byte access moves a unit and half
// as many lanes cover a row as with RowIO, so a wave holds twice as many
// positives; a packed bf16 unit takes four registers.  The float variant
// (the contributions of repeated rows) keeps the same element ownership.
template <int G, int U, typename E>
struct PairIO;

template <int G, int U>
struct PairIO<G, U, bf16_t> {
    static constexpr int C = 2 * U;
    using Elem = bf16_t;
    using Reg = uint4;
    static constexpr int R = U;
    __device__ __forceinline__ static void load_packed(Reg (&r)[R],
                                                       const bf16_t* __restrict__ base,
                                                       int64_t row, int32_t D, int lane) {
        const uint4* p = reinterpret_cast<const uint4*>(base + row * (int64_t)D);
        const int nu = D >> 3;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = lane + u * G;
            r[u] = (k < nu) ? p[k] : make_uint4(0u, 0u, 0u, 0u);
        }
    }
    __device__ __forceinline__ static float4 chunk(const Reg (&r)[R], int c) {
        const uint4 w = r[c >> 1];
        return bf16x4_to_float4((c & 1) ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y));
    }
    __device__ __forceinline__ static void refresh(Reg (&r)[R]) {
#pragma unroll
        for (int u = 0; u < R; ++u)
            asm volatile("" : "+v"(r[u].x), "+v"(r[u].y), "+v"(r[u].z), "+v"(r[u].w));
    }
    __device__ __forceinline__ static void load(float4 (&x)[C], const bf16_t* __restrict__ base,
                                                int64_t row, int32_t D, int lane) {
        Reg r[R];
        load_packed(r, base, row, D, lane);
#pragma unroll
        for (int c = 0; c < C; ++c) x[c] = chunk(r, c);
    }
    __device__ __forceinline__ static void store(bf16_t* __restrict__ base, int64_t row,
                                                 int32_t D, int lane, const float4 (&x)[C]) {
        uint4* p = reinterpret_cast<uint4*>(base + row * (int64_t)D);
        const int nu = D >> 3;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = lane + u * G;
            if (k < nu) {
                const uint2 a = float4_to_bf16x4(x[2 * u]), b = float4_to_bf16x4(x[2 * u + 1]);
                p[k] = make_uint4(a.x, a.y, b.x, b.y);
            }
        }
    }
    __device__ __forceinline__ static float dot(const float4 (&a)[C], const float4 (&b)[C]) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < C; ++c) s += dot4(a[c], b[c]);
        return s;
    }
    __device__ __forceinline__ static float dotp(const float4 (&a)[C], const Reg (&b)[R]) {
        float s = 0.f;
#pragma unroll
        for (int c = 0; c < C; ++c) s += dot4(a[c], chunk(b, c));
        return s;
    }
};

template <int G, int U>
struct PairIO<G, U, float> {
    static constexpr int C = 2 * U;
    using Elem = float;
    using Reg = float4;
    static constexpr int R = 2 * U;
    __device__ __forceinline__ static void load_packed(Reg (&r)[R], const float* __restrict__ base,
                                                       int64_t row, int32_t D, int lane) {
        const float4* p = reinterpret_cast<const float4*>(base + row * (int64_t)D);
        const int nu = D >> 3;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int k = lane + (c >> 1) * G;
            r[c] = (k < nu) ? p[2 * k + (c & 1)] : zero4();
        }
    }
    __device__ __forceinline__ static float4 chunk(const Reg (&r)[R], int c) { return r[c]; }
    __device__ __forceinline__ static void refresh(Reg (&)[R]) {}
    __device__ __forceinline__ static void load(float4 (&x)[C], const float* __restrict__ base,
                                                int64_t row, int32_t D, int lane) {
        load_packed(x, base, row, D, lane);
    }
    __device__ __forceinline__ static void store(float* __restrict__ base, int64_t row, int32_t D,
                                                 int lane, const float4 (&x)[C]) {
        float4* p = reinterpret_cast<float4*>(base + row * (int64_t)D);
        const int nu = D >> 3;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int k = lane + (c >> 1) * G;
            if (k < nu) p[2 * k + (c & 1)] = x[c];
        }
    }
};

// Record the first error since the last huge_check and flag this call.
// Weight c_i of positive i: its float weight where weights are given, else
// its integer co_count.
__device__ __forceinline__ float positive_weight(const StepArgs& a, int64_t i) {
    return a.w != nullptr ? a.w[i] : (float)a.cc[i];
}

// A usable weight: finite and >= 0 (a co_count >= 0).
__device__ __forceinline__ bool weight_valid(const StepArgs& a, int64_t i) {
    if (a.w != nullptr) {
        const float c = a.w[i];
        return c >= 0.f && c <= 3.402823466e38f;
    }
    return a.cc[i] >= 0;
}

__device__ __forceinline__ void raise_error(Control* ctl, uint32_t bit) {
    atomicOr(&ctl->step_bad, bit);
    atomicCAS(&ctl->error, 0u, bit);
}

// A failed internal check: flags the call and records which check failed.
__device__ __forceinline__ void raise_internal(Control* ctl, uint32_t site) {
    raise_error(ctl, kBadInternal);
    atomicCAS(&ctl->site, 0u, site);
}

}  // namespace huge
