// Co-occurrence triples from uniform random walks on a CSR graph in device
// memory: the sampler that produces the training step's input (HUGE
// Sec. 3.2, Alg. 1), on the GPU.
//
// Every seed node s is repeated gamma times; walk r of s takes k uniform
// steps: w_0 = s, and w_t is neighbour floor(x deg / 2^64) of w_{t-1}, with x
// the first 64 bits of Philox4x32-10 on counter (lo32 s, hi32 s, r, 4 + t); a
// node without neighbours ends the walk.  The walks of one seed are grouped
// and their co-occurrences combined (Alg. 1, GroupByKey and CombineValues):
// the pairs (s, w_t) for t <= window, or -- DeepWalk's window -- every ordered
// pair (w_a, w_b) of a walk with 1 <= |a - b| <= window; pairs of a node with
// itself are dropped.  One triple per distinct (source, destination) of a
// seed: cc = its co-occurrences, hist[d - 1] = those at distance d.  Seeds are
// emitted in ascending order and, within a seed, (source, destination)
// ascending, so the output is bitwise reproducible.
//
// One workgroup per seed: the walks go to LDS, their pairs to LDS as 64-bit
// keys (source << 32 | destination) with the distance beside them, a bitonic
// sort groups equal keys, and each run becomes a triple.  A counting pass and
// an exclusive scan of the per-seed counts place every seed's triples; the
// writing pass repeats the (deterministic) walks.
#include "common.hpp"
#include "device.hpp"

namespace huge {

// Sum over the workgroup (kBlock threads) of one value per thread: returns
// the exclusive prefix of this thread, *total gets the sum.  Synchronises.
__device__ __forceinline__ uint32_t walk_block_excl(uint32_t v, uint32_t* s_tmp,
                                                    uint32_t* total) {
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

// Walk r of seed s into w[0 .. k]; returns the last position reached, or -1
// (and reports) if the graph is malformed.
__device__ int32_t do_walk(const WalkArgs& A, int64_t s, int32_t r, int32_t* w,
                           int32_t* status) {
    w[0] = (int32_t)s;
    const uint32_t key_lo = (uint32_t)A.seed, key_hi = (uint32_t)(A.seed >> 32);
    int64_t cur = s;
    for (int32_t t = 1; t <= A.steps; ++t) {
        const int64_t b = A.off[cur], e = A.off[cur + 1];
        if (b < 0 || e < b || e > A.num_edges) {
            atomicCAS(status, 0, -2);
            return -1;
        }
        const uint64_t deg = (uint64_t)(e - b);
        if (deg == 0) return t - 1;
        const uint4 rr = philox4x32_10(
            make_uint4((uint32_t)s, (uint32_t)((uint64_t)s >> 32), (uint32_t)r, 4u + (uint32_t)t),
            key_lo, key_hi);
        const uint64_t x = ((uint64_t)rr.y << 32) | (uint64_t)rr.x;
        const int64_t next = A.nbr[b + (int64_t)__umul64hi(x, deg)];
        if (next < 0 || next >= A.num_nodes) {
            atomicCAS(status, 0, -2);
            return -1;
        }
        w[t] = (int32_t)next;
        cur = next;
    }
    return A.steps;
}

// Pairs of one walk (positions 0 .. last), in loop order; emit(key, dist) for
// each, returns their number.
template <typename Emit>
__device__ __forceinline__ uint32_t walk_pairs(const WalkArgs& A, const int32_t* w, int32_t last,
                                               Emit emit) {
    uint32_t c = 0;
    for (int32_t a = 0; a <= last; ++a) {
        if (A.seed_only && a > 0) break;
        const int32_t b0 = A.seed_only ? a + 1 : (a - A.window > 0 ? a - A.window : 0);
        const int32_t b1 = a + A.window < last ? a + A.window : last;
        for (int32_t b = b0; b <= b1; ++b) {
            if (b == a || w[a] == w[b]) continue;
            emit(((uint64_t)(uint32_t)w[a] << 32) | (uint64_t)(uint32_t)w[b],
                 (uint32_t)(a > b ? a - b : b - a));
            ++c;
        }
    }
    return c;
}

// One kernel for both passes: WRITE = false stores the number of triples of
// each seed in counts[g]; WRITE = true writes them from offsets[g].
template <bool WRITE>
__global__ __launch_bounds__(kBlock) void k_walk(WalkArgs A, uint32_t* __restrict__ counts,
                                                 const uint64_t* __restrict__ offsets,
                                                 const int64_t* __restrict__ total,
                                                 int64_t capacity, int32_t* __restrict__ src,
                                                 int32_t* __restrict__ dst,
                                                 int32_t* __restrict__ cc,
                                                 int32_t* __restrict__ hist,
                                                 int32_t* __restrict__ status) {
    __shared__ int32_t s_walk[kWalkMaxNodes];
    __shared__ uint64_t s_key[kWalkMaxPairs];
    __shared__ uint8_t s_dist[kWalkMaxPairs];
    __shared__ uint32_t s_tmp[2][kBlock / 64];
    __shared__ int32_t s_last[kWalkMaxWalks];
    const int tid = threadIdx.x;
    if (WRITE && (*status != 0 || *total > capacity)) return;  // uniform
    const int32_t W = A.steps + 1;
    for (int64_t g = blockIdx.x; g < A.num_seeds; g += gridDim.x) {
        const int64_t s = A.first_seed + g;
        // walks
        for (int32_t r = tid; r < A.walks; r += kBlock)
            s_last[r] = do_walk(A, s, r, s_walk + (int64_t)r * W, status);
        __syncthreads();
        // pairs: per-thread counts, a block scan, then the pairs at their slots
        uint32_t mine = 0;
        for (int32_t r = tid; r < A.walks; r += kBlock)
            if (s_last[r] > 0)
                mine += walk_pairs(A, s_walk + (int64_t)r * W, s_last[r],
                                   [](uint64_t, uint32_t) {});
        uint32_t np;
        uint32_t at = walk_block_excl(mine, s_tmp[0], &np);
        for (int32_t r = tid; r < A.walks; r += kBlock)
            if (s_last[r] > 0)
                walk_pairs(A, s_walk + (int64_t)r * W, s_last[r], [&](uint64_t key, uint32_t d) {
                    s_key[at] = key;
                    s_dist[at] = (uint8_t)d;
                    ++at;
                });
        // bitonic sort of the keys (padded to a power of two) with their distance
        uint32_t P = 1;
        while (P < np) P <<= 1;
        for (uint32_t i = np + tid; i < P; i += kBlock) {
            s_key[i] = ~0ull;
            s_dist[i] = 0;
        }
        __syncthreads();
        for (uint32_t size = 2; size <= P; size <<= 1) {
            for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
                for (uint32_t i = tid; i < P / 2; i += kBlock) {
                    const uint32_t lo = 2 * i - (i & (stride - 1));
                    const uint32_t hi = lo + stride;
                    const bool up = (lo & size) == 0;
                    const uint64_t a = s_key[lo], b = s_key[hi];
                    if ((a > b) == up) {
                        s_key[lo] = b;
                        s_key[hi] = a;
                        const uint8_t t = s_dist[lo];
                        s_dist[lo] = s_dist[hi];
                        s_dist[hi] = t;
                    }
                }
                __syncthreads();
            }
        }
        // runs of equal keys: thread t owns entries [t * per, (t + 1) * per)
        const uint32_t per = (np + kBlock - 1) / kBlock;
        const uint32_t i0 = tid * per;
        const uint32_t i1 = i0 + per < np ? i0 + per : np;
        uint32_t starts = 0;
        for (uint32_t i = i0; i < i1; ++i)
            if (i == 0 || s_key[i] != s_key[i - 1]) ++starts;
        uint32_t runs;
        uint32_t rank = walk_block_excl(starts, s_tmp[1], &runs);
        if (!WRITE) {
            if (tid == 0) counts[g] = runs;
        } else {
            const uint64_t base = offsets[g];
            for (uint32_t i = i0; i < i1; ++i) {
                if (!(i == 0 || s_key[i] != s_key[i - 1])) continue;
                uint32_t j = i + 1;
                while (j < np && s_key[j] == s_key[i]) ++j;
                const uint64_t o = base + rank;
                ++rank;
                if ((int64_t)o >= capacity) continue;  // cannot happen: the total fits
                src[o] = (int32_t)(s_key[i] >> 32);
                dst[o] = (int32_t)(uint32_t)s_key[i];
                cc[o] = (int32_t)(j - i);
                if (hist != nullptr) {
                    for (int32_t d = 1; d <= A.window; ++d) {
                        int32_t c = 0;
                        for (uint32_t q = i; q < j; ++q) c += s_dist[q] == d ? 1 : 0;
                        hist[(int64_t)o * A.window + (d - 1)] = c;
                    }
                }
            }
        }
        __syncthreads();  // LDS is reused by the next seed
    }
}

// Exclusive scan of the per-seed counts into 64-bit offsets; *total gets the
// number of triples.  One workgroup; it also clears the status word first.
__global__ __launch_bounds__(kBlock) void k_walk_scan(const uint32_t* __restrict__ counts,
                                                      uint64_t* __restrict__ offsets, int64_t n,
                                                      int64_t* __restrict__ total) {
    __shared__ uint32_t s_tmp[kBlock / 64];
    __shared__ uint64_t s_carry;
    if (threadIdx.x == 0) s_carry = 0;
    __syncthreads();
    constexpr int kPer = 8;
    for (int64_t c0 = 0; c0 < n; c0 += (int64_t)kBlock * kPer) {
        uint32_t v[kPer];
        uint32_t sum = 0;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t i = c0 + (int64_t)threadIdx.x * kPer + q;
            v[q] = i < n ? counts[i] : 0u;
            sum += v[q];
        }
        uint32_t chunk;
        uint32_t ex = walk_block_excl(sum, s_tmp, &chunk);
        const uint64_t carry = s_carry;
        uint64_t run = carry + ex;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int64_t i = c0 + (int64_t)threadIdx.x * kPer + q;
            if (i < n) offsets[i] = run;
            run += v[q];
        }
        __syncthreads();
        if (threadIdx.x == 0) s_carry = carry + chunk;
        __syncthreads();
    }
    if (threadIdx.x == 0) *total = (int64_t)s_carry;
}

__global__ void k_walk_begin(int32_t* status) {
    if (threadIdx.x == 0) *status = 0;
}

// After the scan: a total above the capacity is reported (nothing is written).
__global__ void k_walk_capacity(const int64_t* total, int64_t capacity, int32_t* status) {
    if (threadIdx.x == 0 && *status == 0 && *total > capacity) *status = -4;
}

hipError_t launch_walks(const WalkArgs& A, uint32_t* counts, uint64_t* offsets, int64_t* total,
                        int64_t capacity, int32_t* src, int32_t* dst, int32_t* cc, int32_t* hist,
                        int32_t* status, hipStream_t s) {
    hipLaunchKernelGGL(k_walk_begin, dim3(1), dim3(64), 0, s, status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || A.num_seeds == 0) {
        if (e == hipSuccess) {
            hipLaunchKernelGGL(k_walk_scan, dim3(1), dim3(kBlock), 0, s, counts, offsets,
                               (int64_t)0, total);
            e = hipGetLastError();
        }
        return e;
    }
    const int64_t grid = A.num_seeds < 65536 ? A.num_seeds : 65536;
    hipLaunchKernelGGL(k_walk<false>, dim3((unsigned)grid), dim3(kBlock), 0, s, A, counts,
                       nullptr, nullptr, capacity, nullptr, nullptr, nullptr, nullptr, status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_walk_scan, dim3(1), dim3(kBlock), 0, s, counts, offsets, A.num_seeds,
                       total);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_walk_capacity, dim3(1), dim3(64), 0, s, total, capacity, status);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_walk<true>, dim3((unsigned)grid), dim3(kBlock), 0, s, A, counts,
                       offsets, total, capacity, src, dst, cc, hist, status);
    return hipGetLastError();
}

}  // namespace huge
