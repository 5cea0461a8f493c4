// Grouping of the rows a batch touches: a stable LSD radix sort of the
// occurrence keys (one kernel per digit of 8 to 10 bits, single pass over the
// data with decoupled look-back between tiles), then run marking on the
// sorted keys.
//
// Occurrence o = i (2 + K) + slot of positive i carries key N + src (slot 0,
// source table) or the context row id (destination, negatives).  After the
// sort, equal keys are adjacent and, the sort being stable, in occurrence
// order: that is the order in which repeated rows sum their contributions.
#include "common.hpp"
#include "device.hpp"

namespace huge {

// Look-back word: [tag:30 | flag:2 | count:32].  The tag identifies the
// (call, pass); words of earlier calls read as "not yet published".
constexpr uint64_t kFlagAggregate = 1ull;
constexpr uint64_t kFlagPrefix = 2ull;

__device__ __forceinline__ uint64_t lb_word(uint32_t tag, uint64_t flag, uint32_t count) {
    return ((uint64_t)(tag & 0x3FFFFFFFu) << 34) | (flag << 32) | (uint64_t)count;
}

__device__ __forceinline__ void lb_store(uint64_t* p, uint64_t w) {
    __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ uint64_t lb_load(const uint64_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Inclusive sum over the first kBins threads of the workgroup (one value
// each): wave shuffles, then the wave totals through LDS.  Every thread of
// the workgroup must call it (it synchronises); the others get 0.
template <int kBins>
__device__ __forceinline__ uint32_t digit_inclusive_sum(uint32_t v, uint32_t* s_tmp) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const bool mine = threadIdx.x < kBins;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(v, off, 64);
        if (lane >= off) v += t;
    }
    if (mine && lane == 63) s_tmp[wave] = v;
    __syncthreads();
    uint32_t add = 0;
    if (mine)
        for (int w = 0; w < wave; ++w) add += s_tmp[w];
    return mine ? v + add : 0u;
}

// One pass of BITS bits at shift BITS * pass over a tile of kSortTile
// consecutive items, kSortThreads threads; wave w owns items
// [w * 512, (w + 1) * 512) of the tile in kSortItems rounds of 64.
//   rank:    lanes of a round holding the same digit are found with BITS
//            ballots; one lane per digit adds the round's count to the wave's
//            LDS counter, whose old value places the round after the earlier
//            ones;
//   publish: per digit (threads < 2^BITS), the tile's count; the items are
//            then written to LDS in digit order (stable);
//   look-back: the counts of earlier tiles, kLookBatch words at a time, up
//            to the first inclusive prefix;
//   write:   LDS position p goes to global position p + (digit's global
//            offset - digit's tile offset): runs of equal digits are
//            contiguous, so the writes coalesce.
template <int BITS>
__global__ __launch_bounds__(kSortThreads) void k_radix_pass(
    Control* __restrict__ ctl, uint32_t* __restrict__ tickets,
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t m, int pass,
    const uint32_t* __restrict__ hist, uint64_t* __restrict__ status, uint32_t tag,
    const uint32_t* __restrict__ gate, uint32_t* __restrict__ bstart) {
    constexpr int kBins = 1 << BITS;
    static_assert(kBins <= kSortThreads, "one thread per digit");
    constexpr int kWaves = kSortThreads / 64;
    constexpr int kWaveItems = kSortTile / kWaves;
    __shared__ uint32_t s_wave[kWaves][kBins];
    __shared__ int32_t s_delta[kBins];
    __shared__ uint32_t s_tmp[2][kBins / 64];
    __shared__ uint32_t s_tile;
    __shared__ uint32_t s_keys[kSortTile];
    __shared__ uint32_t s_vals[kSortTile];

    if (ctl->step_bad) return;  // uniform: the call is a no-op
    if (gate != nullptr && *gate == 0u) return;  // the bucket sort completed the order

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int shift = pass * BITS;
    const bool digit_thread = tid < kBins;
    const int d = tid;  // the digit of threads < kBins

    for (int j = tid; j < kWaves * kBins; j += kSortThreads) (&s_wave[0][0])[j] = 0u;
    if (tid == 0) s_tile = atomicAdd(tickets, 1u);
    // Tiles are normally handed out in workgroup order: load that tile's
    // items while the ticket is in flight, reload if it differs.
    uint32_t key[kSortItems], val[kSortItems];
    auto load_tile = [&](int64_t t) {
        const int64_t base = t * kSortTile + (int64_t)wave * kWaveItems;
#pragma unroll
        for (int r = 0; r < kSortItems; ++r) {
            const int64_t idx = base + r * 64 + lane;
            const bool valid = idx < m;
            key[r] = valid ? keys_in[idx] : 0u;
            val[r] = valid ? (vals_in ? vals_in[idx] : (uint32_t)idx) : 0u;
        }
    };
    load_tile(blockIdx.x);
    const uint32_t hd = digit_thread ? hist[d] : 0u;
    const uint32_t global_excl = digit_inclusive_sum<kBins>(hd, s_tmp[0]) - hd;  // synchronises
    const int64_t tile = s_tile;
    if (tile >= (int64_t)gridDim.x) {  // tickets were not reset: refuse, never wait
        if (tid == 0) raise_error(ctl, kBadInternal);
        return;
    }
    if (bstart != nullptr && tile == 0 && digit_thread) bstart[d] = global_excl;
    if (tile != (int64_t)blockIdx.x) load_tile(tile);
    const int64_t base_idx = tile * kSortTile + (int64_t)wave * kWaveItems;

    uint32_t rank[kSortItems];
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    {
        uint32_t before[kSortItems], old[kSortItems];
        int leader[kSortItems];
#pragma unroll
        for (int r = 0; r < kSortItems; ++r) {
            const bool valid = base_idx + r * 64 + lane < m;
            const uint32_t dg = (key[r] >> shift) & (kBins - 1);
            uint64_t peers = __ballot(valid);
#pragma unroll
            for (int b = 0; b < BITS; ++b) {
                const bool bit = (dg >> b) & 1u;
                const uint64_t ones = __ballot(bit);
                peers &= bit ? ones : ~ones;
            }
            before[r] = (uint32_t)__popcll(peers & lt_mask);
            const int ld = __ffsll((long long)peers) - 1;
            leader[r] = ld < 0 ? 0 : ld;
            old[r] = 0u;
            if (valid && before[r] == 0)
                old[r] = atomicAdd(&s_wave[wave][dg], (uint32_t)__popcll(peers));
        }
#pragma unroll
        for (int r = 0; r < kSortItems; ++r) rank[r] = __shfl(old[r], leader[r], 64) + before[r];
    }
    __syncthreads();

    // Per digit: wave offsets, tile count, publication.
    uint32_t tile_count = 0;
    uint32_t wcnt[kWaves];
    if (digit_thread) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            wcnt[w] = s_wave[w][d];
            tile_count += wcnt[w];
        }
        lb_store(status + tile * kBins + d,
                 lb_word(tag, tile == 0 ? kFlagPrefix : kFlagAggregate, tile_count));
    }
    const uint32_t local_excl = digit_inclusive_sum<kBins>(tile_count, s_tmp[1]) - tile_count;
    if (digit_thread) {
        uint32_t run = local_excl;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            s_wave[w][d] = run;
            run += wcnt[w];
        }
    }
    __syncthreads();

    // Stable tile-local order in LDS.
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        if (base_idx + r * 64 + lane < m) {
            const uint32_t dg = (key[r] >> shift) & (kBins - 1);
            const uint32_t p = s_wave[wave][dg] + rank[r];
            s_keys[p] = key[r];
            s_vals[p] = val[r];
        }
    }

    // Decoupled look-back over the tiles before this one, for digit d.
    if (digit_thread) {
        uint32_t excl = 0;
        if (tile > 0) {
            const uint32_t want = tag & 0x3FFFFFFFu;
            int64_t look = tile - 1;
            uint32_t spins = 0;
            bool done = false;
            while (!done) {
                uint64_t w[kLookBatch];
#pragma unroll
                for (int j = 0; j < kLookBatch; ++j)
                    w[j] = (look - j >= 0) ? lb_load(status + (look - j) * kBins + d)
                                           : lb_word(want, kFlagPrefix, 0u);
                int used = 0;
                bool stop = false;
#pragma unroll
                for (int j = 0; j < kLookBatch; ++j) {
                    if (!stop) {
                        const uint64_t flag = (w[j] >> 32) & 3ull;
                        if ((uint32_t)(w[j] >> 34) != want || flag == 0ull) {
                            stop = true;
                        } else {
                            excl += (uint32_t)w[j];
                            used = j + 1;
                            if (flag == kFlagPrefix) {
                                done = true;
                                stop = true;
                            }
                        }
                    }
                }
                look -= used;
                if (!done && used < kLookBatch) {
                    // every earlier tile is resident (it holds a smaller
                    // ticket) and publishes without waiting; the bound only
                    // guards against a broken invariant, turning it into a
                    // reported error
                    if (++spins > (1u << 22)) {
                        raise_error(ctl, kBadInternal);
                        break;
                    }
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            lb_store(status + tile * kBins + d,
                     lb_word(tag, kFlagPrefix, excl + tile_count));
        }
        s_delta[d] = (int32_t)(global_excl + excl) - (int32_t)local_excl;
    }
    __syncthreads();

    const int64_t tile_base = tile * kSortTile;
    const int64_t valid_n = (m - tile_base) < kSortTile ? (m - tile_base) : kSortTile;
    for (int p = tid; p < valid_n; p += kSortThreads) {
        const uint32_t k = s_keys[p];
        const int64_t dest = (int64_t)s_delta[(k >> shift) & (kBins - 1)] + p;
        if (dest >= 0 && dest < m) {
            keys_out[dest] = k;
            vals_out[dest] = s_vals[p];
        } else {
            raise_error(ctl, kBadInternal);
        }
    }
}

hipError_t launch_radix_pass(Control* ctl, const uint32_t* keys_in, const uint32_t* vals_in,
                             uint32_t* keys_out, uint32_t* vals_out, int64_t m, int pass,
                             int bits, const uint32_t* hist, uint64_t* status, uint32_t tag,
                             const uint32_t* gate, uint32_t* bstart, hipStream_t s) {
    const int64_t tiles = (m + kSortTile - 1) / kSortTile;
    if (tiles == 0) return hipSuccess;
    if (pass < 0 || pass >= kMaxPasses) return hipErrorInvalidValue;
#define HUGE_RADIX_LAUNCH(B)                                                                  \
    hipLaunchKernelGGL(k_radix_pass<B>, dim3((unsigned)tiles), dim3(kSortThreads), 0, s, ctl, \
                       &ctl->tickets[pass], keys_in, vals_in, keys_out, vals_out, m, pass,    \
                       hist + pass * kMaxBins, status, tag, gate, bstart)
    switch (bits) {
        case 8: HUGE_RADIX_LAUNCH(8); break;
        case 9: HUGE_RADIX_LAUNCH(9); break;
        case 10: HUGE_RADIX_LAUNCH(10); break;
        default: return hipErrorInvalidValue;
    }
#undef HUGE_RADIX_LAUNCH
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Bucket stage: completion of the grouping inside the buckets of the first
// pass.
//
// After the first radix pass (digit = the lowest `bits` key bits) the items
// of bucket b (digit b) occupy positions [bstart[b], bstart[b] + hist0[b])
// in occurrence order.  One workgroup takes one bucket and makes equal keys
// adjacent, in occurrence order, writing the bucket to the output buffer
// (the input buffer itself, or the other one): a small bucket by hashing its
// keys in LDS (k_bucket_group), a larger one by a stable in-LDS LSD sort on
// key bits [bits, key_bits) (k_bucket_sort_large).  A bucket too large for
// both sets ctl->overflow, and the later global radix passes then sort the
// whole array from the first pass's output.  Either way equal keys end up
// adjacent and in occurrence order, which is all the run marking needs.
// ---------------------------------------------------------------------------
template <int THREADS>
__device__ __forceinline__ uint32_t block_exclusive_sum(uint32_t v, uint32_t* s_tmp) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t t = __shfl_up(incl, off, 64);
        if (lane >= off) incl += t;
    }
    if (lane == 63) s_tmp[wave] = incl;
    __syncthreads();
    uint32_t add = 0;
    for (int w = 0; w < wave; ++w) add += s_tmp[w];
    return add + incl - v;
}

// Sorts `size` (<= THREADS * ITEMS) items of one bucket; wave w holds items
// [w * ITEMS * 64, (w + 1) * ITEMS * 64) in ITEMS rounds of 64 lanes.
template <int THREADS, int ITEMS>
__device__ __forceinline__ void bucket_sort_lds(const uint32_t* keys_in, const uint32_t* vals_in,
                                                uint32_t* keys_out, uint32_t* vals_out,
                                                int64_t start, int size, int lo, int rbits,
                                                uint32_t* s_k, uint32_t* s_v,
                                                uint32_t (*s_cnt)[kLocalBins], uint32_t* s_tmp) {
    constexpr int kWaves = THREADS / 64;
    constexpr int kWaveItems = ITEMS * 64;
    constexpr int kDigitsPer = (kLocalBins + THREADS - 1) / THREADS;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    uint32_t key[ITEMS], val[ITEMS];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
        const int e = wave * kWaveItems + r * 64 + lane;
        key[r] = e < size ? keys_in[start + e] : 0u;
        val[r] = e < size ? vals_in[start + e] : 0u;
    }
    const int npass = (rbits + kLocalMaxBits - 1) / kLocalMaxBits;
    const int width = (rbits + npass - 1) / npass;
    for (int q = 0; q < npass; ++q) {
        const int shift = lo + q * width;
        const int wq = (rbits - q * width) < width ? (rbits - q * width) : width;
        const uint32_t mask = (1u << wq) - 1u;
        const int bins = 1 << wq;
        for (int j = tid; j < kWaves * kLocalBins; j += THREADS) (&s_cnt[0][0])[j] = 0u;
        __syncthreads();
        uint32_t rank[ITEMS];
        {
            uint32_t before[ITEMS], old[ITEMS];
            int leader[ITEMS];
#pragma unroll
            for (int r = 0; r < ITEMS; ++r) {
                const bool valid = wave * kWaveItems + r * 64 + lane < size;
                const uint32_t dg = (key[r] >> shift) & mask;
                uint64_t peers = __ballot(valid);
                for (int b = 0; b < wq; ++b) {
                    const bool bit = (dg >> b) & 1u;
                    const uint64_t ones = __ballot(bit);
                    peers &= bit ? ones : ~ones;
                }
                before[r] = (uint32_t)__popcll(peers & lt_mask);
                const int ld = __ffsll((long long)peers) - 1;
                leader[r] = ld < 0 ? 0 : ld;
                old[r] = 0u;
                if (valid && before[r] == 0)
                    old[r] = atomicAdd(&s_cnt[wave][dg], (uint32_t)__popcll(peers));
            }
#pragma unroll
            for (int r = 0; r < ITEMS; ++r) rank[r] = __shfl(old[r], leader[r], 64) + before[r];
        }
        __syncthreads();
        // digit-major, wave-minor exclusive offsets
        uint32_t tot[kDigitsPer];
        uint32_t mine = 0;
#pragma unroll
        for (int j = 0; j < kDigitsPer; ++j) {
            const int d = tid * kDigitsPer + j;
            uint32_t t = 0;
            if (d < bins)
                for (int w = 0; w < kWaves; ++w) t += s_cnt[w][d];
            tot[j] = t;
            mine += t;
        }
        uint32_t run = block_exclusive_sum<THREADS>(mine, s_tmp);  // synchronises
#pragma unroll
        for (int j = 0; j < kDigitsPer; ++j) {
            const int d = tid * kDigitsPer + j;
            if (d < bins) {
                for (int w = 0; w < kWaves; ++w) {
                    const uint32_t c = s_cnt[w][d];
                    s_cnt[w][d] = run;
                    run += c;
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < ITEMS; ++r) {
            if (wave * kWaveItems + r * 64 + lane < size) {
                const uint32_t p = s_cnt[wave][(key[r] >> shift) & mask] + rank[r];
                s_k[p] = key[r];
                s_v[p] = val[r];
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < ITEMS; ++r) {
            const int e = wave * kWaveItems + r * 64 + lane;
            if (e < size) {
                key[r] = s_k[e];
                val[r] = s_v[e];
            }
        }
        __syncthreads();  // s_cnt and s_tmp are reused by the next pass
    }
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
        const int e = wave * kWaveItems + r * 64 + lane;
        if (e < size) {
            keys_out[start + e] = key[r];
            vals_out[start + e] = val[r];
        }
    }
}

constexpr int kBucketLargeThreads = 1024;
constexpr int kBucketLargeItems = 12;   // up to 12288 items per bucket

// ---------------------------------------------------------------------------
// Grouping of one small bucket (at most kGroupCap items) without sorting it:
// equal keys only have to be adjacent and in occurrence order.
//   1. every item inserts its key into an LDS hash table (linear probing)
//      and counts it there;
//   2. items whose key occurs once keep their relative order and fill the
//      front of the bucket (their position = their index minus the number of
//      repeated items before them);
//   3. the repeated items, listed in occurrence order, are placed by one
//      wave: groups in the order of their first occurrence, each in
//      occurrence order.
// The result does not depend on where a key landed in the table.  Larger
// buckets are queued for k_bucket_sort_large.
// ---------------------------------------------------------------------------
constexpr int kGroupThreads = 256;
constexpr int kGroupItems = 8;                              // item e = tid * 8 + r
constexpr int kGroupCap = kGroupThreads * kGroupItems;      // 2048
constexpr int kGroupSlotBits = 12;
constexpr int kGroupSlots = 1 << kGroupSlotBits;            // twice the capacity
constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;                 // keys are below 2N <= 2^32 - 2

// keys_in/vals_in may be the same buffers as keys_out/vals_out: every item
// is read before the first write.
__global__ __launch_bounds__(kGroupThreads) void k_bucket_group(
    Control* ctl, const uint32_t* keys_in, const uint32_t* vals_in, uint32_t* keys_out,
    uint32_t* vals_out, int64_t m, int lo, const uint32_t* __restrict__ hist0,
    const uint32_t* __restrict__ bstart, uint32_t* __restrict__ biglist) {
    __shared__ uint32_t s_slot_key[kGroupSlots];     // table keys; later the group states
    __shared__ uint32_t s_count[kGroupSlots / 2];    // two 16-bit counts per word
    __shared__ uint32_t s_rep[kGroupCap];            // repeated items: slot << 16 | e
    __shared__ uint16_t s_pos[kGroupCap];            // final position of repeated item e
    __shared__ uint32_t s_tmp[kGroupThreads / 64];
    if (ctl->step_bad) return;
    const int b = blockIdx.x;
    const uint32_t size = hist0[b];
    if (size == 0u) return;
    if (size > (uint32_t)kGroupCap) {
        if (threadIdx.x == 0) biglist[atomicAdd(&ctl->big_count, 1u)] = (uint32_t)b;
        return;
    }
    const int64_t start = bstart[b];
    if (start + (int64_t)size > m) {
        if (threadIdx.x == 0) raise_error(ctl, kBadInternal);
        return;
    }
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int n = (int)size;
    for (int j = tid; j < kGroupSlots; j += kGroupThreads) s_slot_key[j] = kEmptyKey;
    for (int j = tid; j < kGroupSlots / 2; j += kGroupThreads) s_count[j] = 0u;
    uint32_t key[kGroupItems], val[kGroupItems], slot[kGroupItems];
#pragma unroll
    for (int r = 0; r < kGroupItems; ++r) {
        const int e = tid * kGroupItems + r;
        key[r] = e < n ? keys_in[start + e] : 0u;
        val[r] = e < n ? vals_in[start + e] : 0u;
    }
    __syncthreads();
    // 1. insert and count.  The table has more slots than the bucket has
    //    items, so every probe sequence ends at the key or at an empty slot.
#pragma unroll
    for (int r = 0; r < kGroupItems; ++r) {
        slot[r] = 0u;
        if (tid * kGroupItems + r < n) {
            uint32_t h = ((key[r] >> lo) * 0x9E3779B1u) >> (32 - kGroupSlotBits);
            for (int probe = 0; probe < kGroupSlots; ++probe) {
                const uint32_t old = atomicCAS(&s_slot_key[h], kEmptyKey, key[r]);
                if (old == kEmptyKey || old == key[r]) break;
                h = (h + 1u) & (uint32_t)(kGroupSlots - 1);
            }
            slot[r] = h;
            atomicAdd(&s_count[h >> 1], 1u << ((h & 1u) * 16u));
        }
    }
    __syncthreads();
    // 2. repeated items before each item (block scan over threads); the
    //    others are written now
    uint32_t rep_mask = 0u, nrep = 0u;
#pragma unroll
    for (int r = 0; r < kGroupItems; ++r) {
        if (tid * kGroupItems + r < n) {
            const uint32_t c = (s_count[slot[r] >> 1] >> ((slot[r] & 1u) * 16u)) & 0xFFFFu;
            if (c > 1u) {
                rep_mask |= 1u << r;
                ++nrep;
            }
        }
    }
    const uint32_t rep_before = block_exclusive_sum<kGroupThreads>(nrep, s_tmp);  // synchronises
    uint32_t rep_total = 0;
    for (int w = 0; w < kGroupThreads / 64; ++w) rep_total += s_tmp[w];
    const uint32_t uniq_total = (uint32_t)n - rep_total;
    {
        uint32_t k = rep_before;
#pragma unroll
        for (int r = 0; r < kGroupItems; ++r) {
            const int e = tid * kGroupItems + r;
            if (e < n) {
                if (rep_mask & (1u << r)) {
                    s_rep[k++] = (slot[r] << 16) | (uint32_t)e;
                } else {
                    const int64_t dst = start + (int64_t)((uint32_t)e - k);
                    keys_out[dst] = key[r];
                    vals_out[dst] = val[r];
                }
            }
        }
    }
    __syncthreads();  // every item has read its count; the table keys are no longer needed
    for (int j = tid; j < kGroupSlots; j += kGroupThreads) s_slot_key[j] = kEmptyKey;
    __syncthreads();
    // 3. one wave places the repeated items; s_slot_key[slot] becomes the
    //    group state (first position << 16 | items placed so far)
    if (wave == 0 && rep_total > 0u) {
        const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        uint32_t gsum = 0u;  // items of the groups started so far
        for (uint32_t j0 = 0; j0 < rep_total; j0 += 64) {
            const uint32_t j = j0 + (uint32_t)lane;
            const bool act = j < rep_total;
            const uint32_t ent = act ? s_rep[j] : 0u;
            const uint32_t sl = ent >> 16, e = ent & 0xFFFFu;
            uint64_t peers = __ballot(act);
#pragma unroll
            for (int bt = 0; bt < kGroupSlotBits; ++bt) {
                const bool bit = (sl >> bt) & 1u;
                const uint64_t ones = __ballot(bit);
                peers &= bit ? ones : ~ones;
            }
            const uint32_t before = (uint32_t)__popcll(peers & lt_mask);
            const int ld = __ffsll((long long)peers) - 1;
            const int leader = ld < 0 ? 0 : ld;
            const bool is_leader = act && before == 0u;
            const uint32_t st = is_leader ? s_slot_key[sl] : 0u;
            const bool starts = is_leader && st == kEmptyKey;
            const uint32_t c = starts ? (s_count[sl >> 1] >> ((sl & 1u) * 16u)) & 0xFFFFu : 0u;
            uint32_t incl = c;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const uint32_t t = __shfl_up(incl, off, 64);
                if (lane >= off) incl += t;
            }
            uint32_t base = starts ? gsum + incl - c : (st >> 16);
            uint32_t placed = starts ? 0u : (st & 0xFFFFu);
            if (is_leader) s_slot_key[sl] = (base << 16) | (placed + (uint32_t)__popcll(peers));
            base = __shfl(base, leader, 64);
            placed = __shfl(placed, leader, 64);
            if (act) s_pos[e] = (uint16_t)(uniq_total + base + placed + before);
            gsum += __shfl(incl, 63, 64);
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kGroupItems; ++r) {
        if (rep_mask & (1u << r)) {
            const int e = tid * kGroupItems + r;
            const uint32_t pos = s_pos[e];
            if (pos >= uniq_total && pos < (uint32_t)n) {
                keys_out[start + (int64_t)pos] = key[r];
                vals_out[start + (int64_t)pos] = val[r];
            } else {
                raise_error(ctl, kBadInternal);
            }
        }
    }
}

// Buckets queued by the small kernel; a fixed grid walks the queue.
__global__ __launch_bounds__(kBucketLargeThreads) void k_bucket_sort_large(
    Control* ctl, const uint32_t* keys_in, const uint32_t* vals_in, uint32_t* keys_out,
    uint32_t* vals_out, int64_t m, int lo, int rbits, const uint32_t* __restrict__ hist0,
    const uint32_t* __restrict__ bstart, const uint32_t* __restrict__ biglist, int bins) {
    constexpr int kCap = kBucketLargeThreads * kBucketLargeItems;
    __shared__ uint32_t s_k[kCap], s_v[kCap];
    __shared__ uint32_t s_cnt[kBucketLargeThreads / 64][kLocalBins];
    __shared__ uint32_t s_tmp[kBucketLargeThreads / 64];
    if (ctl->step_bad) return;
    const uint32_t count = ctl->big_count;
    for (uint32_t q = blockIdx.x; q < count && q < (uint32_t)bins; q += gridDim.x) {
        const uint32_t b = biglist[q];
        if (b >= (uint32_t)bins) {
            if (threadIdx.x == 0) raise_error(ctl, kBadInternal);
            return;
        }
        const uint32_t size = hist0[b];
        if (size > (uint32_t)kCap) {  // the later global passes sort everything
            if (threadIdx.x == 0) atomicOr(&ctl->overflow, 1u);
            continue;
        }
        const int64_t start = bstart[b];
        if (start + (int64_t)size > m) {
            if (threadIdx.x == 0) raise_error(ctl, kBadInternal);
            return;
        }
        bucket_sort_lds<kBucketLargeThreads, kBucketLargeItems>(
            keys_in, vals_in, keys_out, vals_out, start, (int)size, lo, rbits, s_k, s_v, s_cnt,
            s_tmp);
        __syncthreads();  // LDS is reused by the next bucket
    }
}

hipError_t launch_bucket_sort(Control* ctl, const uint32_t* keys_in, const uint32_t* vals_in,
                              uint32_t* keys_out, uint32_t* vals_out, int64_t m, int bits,
                              int key_bits, const uint32_t* hist0, const uint32_t* bstart,
                              uint32_t* biglist, hipStream_t s) {
    const int rbits = key_bits - bits;
    if (m == 0 || rbits <= 0) return hipSuccess;
    if (bits < 1 || bits > kMaxDigitBits || rbits > 32 - bits) return hipErrorInvalidValue;
    const int bins = 1 << bits;
    hipLaunchKernelGGL(k_bucket_group, dim3((unsigned)bins), dim3(kGroupThreads), 0, s, ctl,
                       keys_in, vals_in, keys_out, vals_out, m, bits, hist0, bstart, biglist);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int grid = bins < 256 ? bins : 256;
    hipLaunchKernelGGL(k_bucket_sort_large, dim3((unsigned)grid), dim3(kBucketLargeThreads), 0, s,
                       ctl, keys_in, vals_in, keys_out, vals_out, m, bits, rbits, hist0, bstart,
                       biglist, bins);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Run marking on the sorted keys, one workgroup per window of kChunk sorted
// positions.  Position j (occurrence o = vals[j]):
//   if its key occurs more than once, info[o] = j (its slot in the duplicate
//   buffer); the sampler has set every entry of the batch to -1.  Runs of a repeated key are cut into pieces at window
//   boundaries; each piece becomes a work item {start, len, key, kind} stored
//   in its window's slots work[w * kChunk ..]:
//     kind 0: the whole run -> sum and update the row directly;
//     kind 1: the run's first piece, the run continues past the window ->
//             partial sum to partB[w]; longhead[w] = its start;
//     kind 2: a later piece, starting at the window boundary -> partA[w].
//   A window holds at most one kind-1 piece.  Per window: number of pieces
//   (with kHasLong set if one is longer than kLongPiece), and {distinct
//   source keys, distinct context keys, repeated occurrences}.
// Everything is written without global atomics.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_mark(const Control* __restrict__ ctl,
                                                 const uint32_t* __restrict__ keys,
                                                 const uint32_t* __restrict__ vals, int64_t m,
                                                 int64_t N, int32_t* __restrict__ info,
                                                 uint4* __restrict__ work,
                                                 uint32_t* __restrict__ wcount,
                                                 uint32_t* __restrict__ longhead,
                                                 uint32_t* __restrict__ wstats) {
    static_assert(kChunk == kBlock, "one workgroup per window");
    __shared__ uint32_t s_cnt[3];
    __shared__ uint32_t s_wave_emit[kBlock / 64];
    __shared__ uint32_t s_long;
    __shared__ uint32_t s_long_piece;
    const int64_t win = blockIdx.x;
    if (ctl->step_bad) {  // unsorted keys: no pieces, nothing marked
        if (threadIdx.x == 0) {
            wcount[win] = 0u;
            longhead[win] = kNoHead;
            wstats[win * 3 + 0] = wstats[win * 3 + 1] = wstats[win * 3 + 2] = 0u;
        }
        return;
    }
    __shared__ uint32_t s_key[kChunk + 2];  // keys j-1 .. window end (inclusive of one past)
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if (tid < 3) s_cnt[tid] = 0u;
    if (tid == 0) {
        s_long = 0xFFFFFFFFu;
        s_long_piece = 0u;
    }
    const int64_t j = win * kChunk + tid;
    // s_key[1 + t] = keys[win * kChunk + t]; s_key[0] = the key before the
    // window, s_key[kChunk + 1] = the key after it (a sentinel if none: it is
    // only compared under an index check)
    s_key[1 + tid] = j < m ? keys[j] : 0u;
    if (tid == 0) s_key[0] = j > 0 ? keys[j - 1] : 0u;
    if (tid == 1) s_key[kChunk + 1] = win * kChunk + kChunk < m ? keys[win * kChunk + kChunk] : 0u;
    __syncthreads();
    bool emit = false, head_S = false, head_T = false, dup = false;
    uint4 rec = make_uint4(0, 0, 0, 0);
    if (j < m) {
        const uint32_t key = s_key[1 + tid];
        const bool prev_same = j > 0 && s_key[tid] == key;
        const bool next_same = j + 1 < m && s_key[2 + tid] == key;
        dup = prev_same || next_same;
        if (dup) {
            const uint32_t o = vals[j];
            if ((int64_t)o < m) info[o] = (int32_t)j;
        }
        head_S = !prev_same && (int64_t)key >= N;
        head_T = !prev_same && (int64_t)key < N;
        if (dup && (!prev_same || tid == 0)) {
            const int64_t win_end = (win + 1) * kChunk;
            const int64_t lim = win_end < m ? win_end : m;
            int64_t e = j + 1;
            while (e < lim && s_key[1 + (e - win * kChunk)] == key) ++e;
            const bool cont_after = (e == win_end) && (e < m) && s_key[kChunk + 1] == key;
            const uint32_t kind = !prev_same ? (cont_after ? 1u : 0u) : 2u;
            rec = make_uint4((uint32_t)j, (uint32_t)(e - j), key, kind);
            emit = true;
            if (kind == 1u) s_long = (uint32_t)j;
        }
    }
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const uint64_t em = __ballot(emit);
    const uint64_t lg = __ballot(emit && rec.y > kLongPiece);
    if (lane == 0 && lg) s_long_piece = 1u;
    const uint64_t bs = __ballot(head_S);
    const uint64_t bt = __ballot(head_T);
    const uint64_t bd = __ballot(dup);
    if (lane == 0) {
        s_wave_emit[wave] = (uint32_t)__popcll(em);
        atomicAdd(&s_cnt[0], (uint32_t)__popcll(bs));
        atomicAdd(&s_cnt[1], (uint32_t)__popcll(bt));
        atomicAdd(&s_cnt[2], (uint32_t)__popcll(bd));
    }
    __syncthreads();
    uint32_t base = 0;
    for (int w = 0; w < wave; ++w) base += s_wave_emit[w];
    if (emit) work[win * kChunk + base + __popcll(em & lt)] = rec;
    if (tid == 0) {
        uint32_t total = 0;
        for (int w = 0; w < kBlock / 64; ++w) total += s_wave_emit[w];
        wcount[win] = total | (s_long_piece ? kHasLong : 0u);
        longhead[win] = s_long;
        wstats[win * 3 + 0] = s_cnt[0];
        wstats[win * 3 + 1] = s_cnt[1];
        wstats[win * 3 + 2] = s_cnt[2];
    }
}

hipError_t launch_mark(Control* ctl, const uint32_t* keys, const uint32_t* vals, int64_t m,
                       int64_t N, int32_t* info, uint4* work, uint32_t* wcount,
                       uint32_t* longhead, uint32_t* wstats, hipStream_t s) {
    const int64_t blocks = (m + kChunk - 1) / kChunk;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_mark, dim3((unsigned)blocks), dim3(kBlock), 0, s, ctl, keys, vals, m, N,
                       info, work, wcount, longhead, wstats);
    return hipGetLastError();
}

}  // namespace huge
