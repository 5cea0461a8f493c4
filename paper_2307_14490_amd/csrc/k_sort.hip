// Grouping of the rows a batch touches (the de-duplication of HUGE Sec. 3.3.2):
// which rows occur once -- those are updated in place by the step -- and, for
// every row that occurs several times, the list of its occurrences in
// occurrence order, which is the order in which its contributions are summed.
//
// Occurrence o = i (2 + K) + slot of positive i carries key N + src (slot 0,
// source table) or the context row id (destination, negatives).
//   1. k_tile_count, k_tile_scan: the occurrences of each digit (lowest 8-10
//      key bits) per tile of kSortTile occurrences, their sums over earlier
//      tiles, and the bucket sizes;
//   2. k_radix_pass: one stable scatter of the occurrences into bucket
//      (digit) order, each bucket in occurrence order; no tile waits for
//      another;
//   3. k_group: one workgroup per bucket finds the bucket's repeated keys,
//      gives every repeated row a contiguous range of duplicate-buffer slots
//      (inside the bucket's own range of positions), writes the slot of each
//      of its occurrences, in occurrence order, to info[o], and lists the
//      repeated rows for the duplicate kernels.
// Steps 1 run with the sampler; the scatter is issued just before the
// previous batch's update and the grouping runs beside that update.
#include "common.hpp"
#include "device.hpp"

namespace huge {

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

// ---------------------------------------------------------------------------
// Digit counts of tile t (kSortTile consecutive keys; kBlock threads,
// coalesced reads): tcount[t * bins + d], digit d = bits [shift, shift + bits)
// of the key.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_tile_count(const Control* __restrict__ ctl,
                                                       const uint32_t* __restrict__ keys,
                                                       int64_t m, int bits, int shift,
                                                       uint32_t* __restrict__ tcount) {
    __shared__ uint32_t s_cnt[kMaxBins];
    const int bins = 1 << bits;
    for (int d = threadIdx.x; d < bins; d += kBlock) s_cnt[d] = 0u;
    __syncthreads();
    const int64_t t = blockIdx.x;
    if (!ctl->step_bad) {
        const int64_t base = t * kSortTile;
        constexpr int kPer = kSortTile / kBlock;
        uint32_t k[kPer];
        bool ok[kPer];
#pragma unroll
        for (int r = 0; r < kPer; ++r) {
            const int64_t o = base + (int64_t)r * kBlock + threadIdx.x;
            ok[r] = o < m;
            k[r] = ok[r] ? keys[o] : 0u;
        }
#pragma unroll
        for (int r = 0; r < kPer; ++r)
            if (ok[r]) atomicAdd(&s_cnt[(k[r] >> shift) & (uint32_t)(bins - 1)], 1u);
    }
    __syncthreads();
    for (int d = threadIdx.x; d < bins; d += kBlock) tcount[t * bins + d] = s_cnt[d];
}

hipError_t launch_tile_count(Control* ctl, const uint32_t* keys, int64_t m, int bits, int shift,
                             uint32_t* tcount, hipStream_t s) {
    const int64_t tiles = (m + kSortTile - 1) / kSortTile;
    if (tiles == 0) return hipSuccess;
    if (bits < kMinDigitBits || bits > kMaxDigitBits || shift < 0 || shift > 31)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_tile_count, dim3((unsigned)tiles), dim3(kBlock), 0, s, ctl, keys, m,
                       bits, shift, tcount);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Per digit d: tprefix[t * bins + d] = sum of tcount[u * bins + d] over tiles
// u < t, and hist[d] = the sum over all tiles.  A workgroup takes
// kScanDigits digits; its kSortThreads / kScanDigits thread groups each sum
// a contiguous range of tiles, and the ranges are combined through LDS.
// ---------------------------------------------------------------------------
constexpr int kScanDigits = 16;
constexpr int kScanGroups = kSortThreads / kScanDigits;  // 64

__global__ __launch_bounds__(kSortThreads) void k_tile_scan(const Control* __restrict__ ctl,
                                                            const uint32_t* __restrict__ tcount,
                                                            int64_t tiles, int bits,
                                                            uint32_t* __restrict__ tprefix,
                                                            uint32_t* __restrict__ hist) {
    __shared__ uint32_t s_part[kScanGroups][kScanDigits];
    if (ctl->step_bad) return;  // uniform
    const int bins = 1 << bits;
    const int dl = threadIdx.x % kScanDigits, g = threadIdx.x / kScanDigits;
    const int d = blockIdx.x * kScanDigits + dl;
    const int64_t per = (tiles + kScanGroups - 1) / kScanGroups;
    const int64_t t0 = (int64_t)g * per;
    const int64_t t1 = t0 + per < tiles ? t0 + per : tiles;
    uint32_t sum = 0;
#pragma unroll 8
    for (int64_t t = t0; t < t1; ++t) sum += tcount[t * bins + d];
    s_part[g][dl] = sum;
    __syncthreads();
    uint32_t run = 0, total = 0;
    for (int h = 0; h < kScanGroups; ++h) {
        const uint32_t v = s_part[h][dl];
        run += h < g ? v : 0u;
        total += v;
    }
    if (g == 0) hist[d] = total;
#pragma unroll 8
    for (int64_t t = t0; t < t1; ++t) {
        const uint32_t v = tcount[t * bins + d];
        tprefix[t * bins + d] = run;
        run += v;
    }
}

hipError_t launch_tile_scan(Control* ctl, const uint32_t* tcount, int64_t m, int bits,
                            uint32_t* tprefix, uint32_t* hist, hipStream_t s) {
    const int64_t tiles = (m + kSortTile - 1) / kSortTile;
    if (tiles == 0) return hipSuccess;
    if (bits < kMinDigitBits || bits > kMaxDigitBits) return hipErrorInvalidValue;
    static_assert((1 << kMinDigitBits) % kScanDigits == 0, "whole digit groups");
    hipLaunchKernelGGL(k_tile_scan, dim3((unsigned)((1 << bits) / kScanDigits)),
                       dim3(kSortThreads), 0, s, ctl, tcount, tiles, bits, tprefix, hist);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Stable scatter by BITS bits at `shift` over a tile of kSortTile
// consecutive items, kSortThreads threads; wave w owns items
// [w * 512, (w + 1) * 512) of the tile in kSortItems rounds of 64.
//   rank:  lanes of a round holding the same digit are found with BITS
//          ballots; one lane per digit adds the round's count to the wave's
//          LDS counter, whose old value places the round after the earlier
//          ones;
//   order: per digit (threads < 2^BITS) the wave offsets; the items are
//          written to LDS in digit order (stable);
//   write: LDS position p goes to global position p + (digit's bucket start
//          + digit's count in earlier tiles - digit's tile offset): runs of
//          equal digits are contiguous, so the writes coalesce.
// vals_out (if not null) receives the position of each key in keys_in.
// ---------------------------------------------------------------------------
template <int BITS>
__global__ __launch_bounds__(kSortThreads) void k_radix_pass(
    Control* __restrict__ ctl, const uint32_t* __restrict__ keys_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t m, int shift,
    const uint32_t* __restrict__ hist, const uint32_t* __restrict__ tprefix,
    uint32_t* __restrict__ bstart) {
    constexpr int kBins = 1 << BITS;
    static_assert(kBins <= kSortThreads, "one thread per digit");
    constexpr int kWaves = kSortThreads / 64;
    constexpr int kWaveItems = kSortTile / kWaves;
    __shared__ uint32_t s_wave[kWaves][kBins];
    __shared__ int32_t s_delta[kBins];
    __shared__ uint32_t s_tmp[2][kBins / 64];
    __shared__ uint32_t s_keys[kSortTile];
    __shared__ uint32_t s_vals[kSortTile];

    if (ctl->step_bad) return;  // uniform: the call is a no-op

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const bool digit_thread = tid < kBins;
    const int d = tid;  // the digit of threads < kBins
    const int64_t tile = blockIdx.x;

    for (int j = tid; j < kWaves * kBins; j += kSortThreads) (&s_wave[0][0])[j] = 0u;
    const int64_t base_idx = tile * kSortTile + (int64_t)wave * kWaveItems;
    uint32_t key[kSortItems];
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t idx = base_idx + r * 64 + lane;
        key[r] = idx < m ? keys_in[idx] : 0u;
    }
    const uint32_t hd = digit_thread ? hist[d] : 0u;
    const uint32_t before_tile = digit_thread ? tprefix[tile * kBins + d] : 0u;
    const uint32_t global_excl = digit_inclusive_sum<kBins>(hd, s_tmp[0]) - hd;  // synchronises
    if (bstart != nullptr && tile == 0 && digit_thread) bstart[d] = global_excl;

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

    // Per digit: wave offsets and the tile's count.
    uint32_t tile_count = 0;
    uint32_t wcnt[kWaves];
    if (digit_thread) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            wcnt[w] = s_wave[w][d];
            tile_count += wcnt[w];
        }
    }
    const uint32_t local_excl = digit_inclusive_sum<kBins>(tile_count, s_tmp[1]) - tile_count;
    if (digit_thread) {
        uint32_t run = local_excl;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            s_wave[w][d] = run;
            run += wcnt[w];
        }
        s_delta[d] = (int32_t)(global_excl + before_tile) - (int32_t)local_excl;
    }
    __syncthreads();

    // Stable tile-local order in LDS.
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t idx = base_idx + r * 64 + lane;
        if (idx < m) {
            const uint32_t p = s_wave[wave][(key[r] >> shift) & (kBins - 1)] + rank[r];
            s_keys[p] = key[r];
            s_vals[p] = (uint32_t)idx;
        }
    }
    __syncthreads();

    const int64_t tile_base = tile * kSortTile;
    const int64_t valid_n = (m - tile_base) < kSortTile ? (m - tile_base) : kSortTile;
    for (int p = tid; p < valid_n; p += kSortThreads) {
        const uint32_t k = s_keys[p];
        const int64_t dest = (int64_t)s_delta[(k >> shift) & (kBins - 1)] + p;
        if (dest >= 0 && dest < m) {
            keys_out[dest] = k;
            if (vals_out != nullptr) vals_out[dest] = s_vals[p];
        } else {
            raise_internal(ctl, kSiteRadixDest);
        }
    }
}

hipError_t launch_radix_pass(Control* ctl, const uint32_t* keys_in, uint32_t* keys_out,
                             uint32_t* vals_out, int64_t m, int bits, int shift,
                             const uint32_t* hist, const uint32_t* tprefix, uint32_t* bstart,
                             hipStream_t s) {
    const int64_t tiles = (m + kSortTile - 1) / kSortTile;
    if (tiles == 0) return hipSuccess;
    if (shift < 0 || shift > 31) return hipErrorInvalidValue;
#define HUGE_RADIX_LAUNCH(B)                                                                  \
    hipLaunchKernelGGL(k_radix_pass<B>, dim3((unsigned)tiles), dim3(kSortThreads), 0, s, ctl, \
                       keys_in, keys_out, vals_out, m, shift, hist, tprefix, bstart)
    switch (bits) {
        case 8: HUGE_RADIX_LAUNCH(8); break;
        case 9: HUGE_RADIX_LAUNCH(9); break;
        case 10: HUGE_RADIX_LAUNCH(10); break;
        default: return hipErrorInvalidValue;
    }
#undef HUGE_RADIX_LAUNCH
    return hipGetLastError();
}

// Exclusive sum of one value per thread over the workgroup (kBlock threads);
// *total receives the sum.  Synchronises; s_tmp holds kBlock / 64 words and
// may be reused after the next barrier.
__device__ __forceinline__ uint32_t block_excl(uint32_t v, uint32_t* s_tmp, uint32_t* total) {
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

// Lanes of the wave whose `bits`-bit value equals this lane's, among the
// lanes in `mask`.
__device__ __forceinline__ uint64_t match_peers(uint32_t value, int bits, uint64_t mask) {
    uint64_t peers = mask;
    for (int b = 0; b < bits; ++b) {
        const bool bit = (value >> b) & 1u;
        const uint64_t ones = __ballot(bit);
        peers &= bit ? ones : ~ones;
    }
    return peers;
}

// ---------------------------------------------------------------------------
// Grouping of one bucket (its items are in occurrence order).
//
// With BM (the bucket's keys differ in at most kBitmapBits bits above the
// bucket digit), a first pass sets, per item, the key's bit in an LDS bitmap
// and, where it was set already, the key's bit in a second bitmap of
// repeated keys; it also counts the bucket's distinct source and destination
// rows.  Only keys marked repeated take part in what follows.
//
// The (repeated) keys are counted in an LDS hash table of 2^TB slots (linear
// probing).  A bucket with more than 3/4 of the slots in distinct keys is
// split into key ranges by further hash bits, each range counted and placed
// in turn (depth first over the binary tree of ranges); at depth 32 a range
// holds one key value, so the split ends.  A count that overflows stops at
// the first chunk that would load the table past 7/8, and the number of
// distinct keys seen so far, scaled to the whole bucket, sets how many levels
// the split descends at once (later sibling ranges start at that depth).
// Per range:
//   count:  every item of the range inserts its key and counts it;
//   emit:   rows counted more than once get consecutive duplicate-buffer
//           slots (positions of the bucket, after those of earlier ranges),
//           and a work record: a short run, a piece, or
//           pieces plus a combine record for a run longer than kPiece;
//   place:  the repeated items, taken in occurrence order (chunk by chunk,
//           compacted, then ranked by one wave 64 at a time), receive their
//           row's next slot: info[o] = slot.
// Where a row's range lands depends on the order of the hash insertions, the
// order of its occurrences does not: every sum is taken in occurrence order.
// Items that occur once keep info = -1 (set by the sampler).
// ---------------------------------------------------------------------------
constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;   // keys are below 2N <= 2^32 - 2
constexpr uint32_t kRepFlag = 0x80000000u;    // table count word: a repeated row, next slot
constexpr int kMaxProbe = 512;                // a longer probe also splits the range

template <int TB>
__device__ __forceinline__ uint32_t slot_hash(uint32_t key) {
    return (key * 0x85EBCA6Bu) >> (32 - TB);
}

__device__ __forceinline__ bool in_range(uint32_t key, int level, uint32_t idx) {
    return level == 0 || ((key * 0xC2B2AE35u) >> (32 - level)) == idx;
}

template <int TB, bool BM>
__global__ __launch_bounds__(kBlock) void k_group(
    Control* __restrict__ ctl, const uint32_t* __restrict__ keys,
    const uint32_t* __restrict__ vals, int64_t m, int64_t N, const uint32_t* __restrict__ hist,
    const uint32_t* __restrict__ bstart, int32_t* __restrict__ info, uint4* __restrict__ shorts,
    uint4* __restrict__ pieces, uint4* __restrict__ combs, ListCaps caps,
    uint32_t* __restrict__ wstats, int bins, int shift, int sub_bits) {
    constexpr int kSlots = 1 << TB;
    constexpr uint32_t kMax = (uint32_t)kSlots / 4u * 3u;    // distinct keys a range may hold
    constexpr uint32_t kLoad = (uint32_t)kSlots / 8u * 7u;   // table load a count stays below
    constexpr int kPer = kSlots / kBlock;                    // table slots per thread
    constexpr int kBitWords = (1 << kBitmapBits) / 32;       // words of one bitmap
    static_assert(!BM || 2 * kSlots <= kBitWords, "the table overlays the first bitmap");
    // the table (key words, then count words); with BM it overlays the bitmap
    // of keys seen, which the table no longer needs, and the bitmap of
    // repeated keys follows
    __shared__ uint32_t s_pool[BM ? 2 * kBitWords : 2 * kSlots];
    uint32_t* const s_key = s_pool;
    uint32_t* const s_cnt = s_pool + kSlots;  // count; after emit, kRepFlag | next slot
    uint32_t* const s_seen = s_pool;
    uint32_t* const s_dup = s_pool + (BM ? kBitWords : 0);
    // repeated items of a chunk in order: their table slot, then their
    // duplicate-buffer slot
    __shared__ uint32_t s_rep[kGroupChunk];
    __shared__ uint32_t s_tmp[6][kBlock / 64];
    __shared__ uint32_t s_distinct, s_fail;
    __shared__ uint32_t s_base[4];
    __shared__ uint32_t s_stat[3];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int b = blockIdx.x; b < bins; b += gridDim.x) {
    __syncthreads();  // LDS of the previous bucket
    if (tid < 3) s_stat[tid] = 0u;
    const uint32_t n = ctl->step_bad ? 0u : hist[b];
    const int64_t s0 = n ? (int64_t)bstart[b] : 0;
    if (n == 0u || s0 + (int64_t)n > m) {
        if (n != 0u && tid == 0) raise_internal(ctl, kSiteGroupBucket);
        if (tid < 3) wstats[b * 3 + tid] = 0u;
        continue;
    }
    const bool single = n <= (uint32_t)kGroupChunk;
    uint32_t key[kGroupItems], val[kGroupItems], slot[kGroupItems];
    auto load_keys = [&](uint32_t c0) {
#pragma unroll
        for (int r = 0; r < kGroupItems; ++r) {
            const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
            key[r] = e < n ? keys[s0 + e] : 0u;
        }
    };
    auto load_chunk = [&](uint32_t c0) {
        load_keys(c0);
#pragma unroll
        for (int r = 0; r < kGroupItems; ++r) {
            const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
            val[r] = e < n ? vals[s0 + e] : 0u;
        }
    };
    if (single) load_chunk(0u);

    // ---- repeated keys (BM) ----
    // the bit of key k is bit (k >> shift) of the bucket's bitmap; a key
    // beyond the bitmap cannot occur (sub_bits <= kBitmapBits)
    const uint32_t bit_words = sub_bits > 5 ? 1u << (sub_bits - 5) : 1u;
    auto repeated = [&](uint32_t k) -> bool {
        if (!BM) return true;
        const uint32_t sub = k >> shift;
        return sub >> 5 < bit_words && ((s_dup[sub >> 5] >> (sub & 31u)) & 1u);
    };
    if (BM) {
        for (uint32_t j = tid; j < bit_words; j += kBlock) {
            s_seen[j] = 0u;
            s_dup[j] = 0u;
        }
        __syncthreads();
        uint32_t nS = 0, nT = 0;
        for (uint32_t c0 = 0; c0 < n; c0 += kGroupChunk) {
            if (!single) load_keys(c0);
#pragma unroll
            for (int r = 0; r < kGroupItems; ++r) {
                const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                if (e >= n) continue;
                const uint32_t sub = key[r] >> shift, w = sub >> 5, bit = 1u << (sub & 31u);
                if (w >= bit_words) {
                    raise_internal(ctl, kSiteGroupBits);
                    continue;
                }
                const uint32_t old = atomicOr(&s_seen[w], bit);
                if (old & bit) {
                    atomicOr(&s_dup[w], bit);
                } else if ((int64_t)key[r] >= N) {
                    ++nS;
                } else {
                    ++nT;
                }
            }
        }
        if (nS) atomicAdd(&s_stat[0], nS);
        if (nT) atomicAdd(&s_stat[1], nT);
        __syncthreads();
    }

    uint32_t rep_base = 0;  // slots handed out to earlier ranges
    int level = 0, depth = 0;  // depth: where the next sibling range starts
    uint32_t ridx = 0;
    while (true) {
        // ---- count ----
        for (int j = tid; j < kSlots; j += kBlock) {
            s_key[j] = kEmptyKey;
            s_cnt[j] = 0u;
        }
        if (tid == 0) {
            s_distinct = 0u;
            s_fail = 0u;
        }
        __syncthreads();
        uint32_t seen = 0;  // items the count went through
        bool over = false;
        for (uint32_t c0 = 0; c0 < n; c0 += kGroupChunk) {
            const uint32_t len = n - c0 < (uint32_t)kGroupChunk ? n - c0 : (uint32_t)kGroupChunk;
            if (s_distinct + len > kLoad) {  // uniform: the table could fill up
                over = true;
                break;
            }
            if (!single) load_chunk(c0);
            // the items of a thread probe together: one compare-and-swap per
            // pending item and step, all issued before any result is used;
            // the counting atomics come after the probe loop
            uint32_t h[kGroupItems], pend = 0u, fresh = 0u;
#pragma unroll
            for (int r = 0; r < kGroupItems; ++r) {
                const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                h[r] = slot_hash<TB>(key[r]);
                if (e < n && in_range(key[r], level, ridx) && repeated(key[r])) pend |= 1u << r;
            }
            uint32_t found = 0u;
            for (int probe = 0; pend != 0u && probe < kMaxProbe; ++probe) {
                uint32_t old[kGroupItems];
#pragma unroll
                for (int r = 0; r < kGroupItems; ++r)
                    old[r] = (pend >> r) & 1u ? atomicCAS(&s_key[h[r]], kEmptyKey, key[r])
                                              : key[r];
#pragma unroll
                for (int r = 0; r < kGroupItems; ++r) {
                    if (!((pend >> r) & 1u)) continue;
                    if (old[r] == kEmptyKey || old[r] == key[r]) {
                        fresh += old[r] == kEmptyKey ? 1u : 0u;
                        found |= 1u << r;
                    } else {
                        h[r] = (h[r] + 1u) & (uint32_t)(kSlots - 1);
                    }
                }
                pend &= ~found;
            }
            if (pend != 0u) s_fail = 1u;
#pragma unroll
            for (int r = 0; r < kGroupItems; ++r) {
                slot[r] = (found >> r) & 1u ? h[r] : kEmptyKey;
                if ((found >> r) & 1u) atomicAdd(&s_cnt[h[r]], 1u);
            }
            if (fresh) atomicAdd(&s_distinct, fresh);
            __syncthreads();
            seen = c0 + len;
            if (s_fail || s_distinct > kMax) {  // uniform
                over = true;
                break;
            }
        }
        if (over) {
            // split the range; its first part next (uniform)
            int add = 1;
            if (!s_fail && seen > 0u) {
                const uint64_t est = (uint64_t)s_distinct * n / seen;
                while (add < 8 && est > ((uint64_t)kMax << add) / 4u * 3u) ++add;
            }
            __syncthreads();
            if (level >= 32) {  // cannot happen: a depth-32 range holds one key value
                if (tid == 0) raise_internal(ctl, kSiteGroupDepth);
                return;
            }
            if (add > 32 - level) add = 32 - level;
            level += add;
            ridx <<= add;
            if (depth < level) depth = level;
            continue;
        }

        // ---- emit ----
        // this thread's table slots (tid, tid + kBlock, ...; conflict-free
        // LDS reads): statistics, slot counts, record counts; slots and
        // records are handed out thread by thread
        uint32_t nS = 0, nT = 0, nrep = 0, nshort = 0, npiece = 0, ncomb = 0, npart = 0;
#pragma unroll 8
        for (int j = 0; j < kPer; ++j) {
            const int q = j * kBlock + tid;
            const uint32_t k = s_key[q];
            if (k == kEmptyKey) continue;
            if (!BM) {  // with BM the first pass counted the rows
                if ((int64_t)k >= N) ++nS; else ++nT;
            }
            const uint32_t c = s_cnt[q];
            if (c > 1u) {
                nrep += c;
                if (c <= kShortRun) {
                    ++nshort;
                } else if (c <= kPiece) {
                    ++npiece;
                } else {
                    const uint32_t np = (c + kPiece - 1) / kPiece;
                    npiece += np;
                    npart += np;
                    ++ncomb;
                }
            }
        }
        uint32_t t_rep, t_short, t_piece, t_comb, t_part;
        uint32_t x_rep = block_excl(nrep, s_tmp[0], &t_rep);
        uint32_t x_short = block_excl(nshort, s_tmp[1], &t_short);
        uint32_t x_piece = block_excl(npiece, s_tmp[2], &t_piece);
        uint32_t x_comb = block_excl(ncomb, s_tmp[3], &t_comb);
        uint32_t x_part = block_excl(npart, s_tmp[4], &t_part);
        if (tid == 0) {
            s_base[0] = t_short ? atomicAdd(&ctl->n_short, t_short) : 0u;
            s_base[1] = t_piece ? atomicAdd(&ctl->n_piece, t_piece) : 0u;
            s_base[2] = t_comb ? atomicAdd(&ctl->n_comb, t_comb) : 0u;
            s_base[3] = t_part ? atomicAdd(&ctl->n_part, t_part) : 0u;
        }
        if (nS) atomicAdd(&s_stat[0], nS);
        if (nT) atomicAdd(&s_stat[1], nT);
        __syncthreads();
        const bool fits = (uint64_t)s_base[0] + t_short <= caps.shorts &&
                          (uint64_t)s_base[1] + t_piece <= caps.pieces &&
                          (uint64_t)s_base[2] + t_comb <= caps.combs &&
                          (uint64_t)s_base[3] + t_part <= caps.parts &&
                          (uint64_t)rep_base + t_rep <= n;
        if (!fits) {  // cannot happen: the capacities bound every batch
            if (tid == 0) raise_internal(ctl, kSiteGroupLists);
            return;
        }
        {
            uint32_t pos = (uint32_t)s0 + rep_base + x_rep;
            uint32_t is = s_base[0] + x_short, ip = s_base[1] + x_piece;
            uint32_t ic = s_base[2] + x_comb, ia = s_base[3] + x_part;
#pragma unroll 4
            for (int j = 0; j < kPer; ++j) {
                const int q = j * kBlock + tid;
                const uint32_t k = s_key[q];
                const uint32_t c = s_cnt[q];
                if (k == kEmptyKey || c <= 1u) continue;
                if (c <= kShortRun) {
                    shorts[is++] = make_uint4(pos, c, k, 0u);
                } else if (c <= kPiece) {
                    pieces[ip++] = make_uint4(pos, c, k, 0u);
                } else {
                    const uint32_t np = (c + kPiece - 1) / kPiece;
                    for (uint32_t z = 0; z < np; ++z) {
                        const uint32_t len = (c - z * kPiece) < kPiece ? (c - z * kPiece) : kPiece;
                        pieces[ip++] = make_uint4(pos + z * kPiece, len, k, ia + z + 1u);
                    }
                    combs[ic++] = make_uint4(k, ia, np, 0u);
                    ia += np;
                }
                s_cnt[q] = kRepFlag | pos;
                pos += c;
            }
        }
        if (tid == 0) s_stat[2] += t_rep;
        __syncthreads();

        // ---- place ----
        if (t_rep > 0u) {
            for (uint32_t c0 = 0; c0 < n; c0 += kGroupChunk) {
                if (!single) {
                    load_chunk(c0);
                    // lookups of the chunk's items, issued together as in the count
                    uint32_t h[kGroupItems], pend = 0u, found = 0u;
#pragma unroll
                    for (int r = 0; r < kGroupItems; ++r) {
                        const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                        h[r] = slot_hash<TB>(key[r]);
                        if (e < n && in_range(key[r], level, ridx) && repeated(key[r]))
                            pend |= 1u << r;
                    }
                    for (int probe = 0; pend != 0u && probe < kMaxProbe; ++probe) {
                        uint32_t cur[kGroupItems];
#pragma unroll
                        for (int r = 0; r < kGroupItems; ++r)
                            cur[r] = (pend >> r) & 1u ? s_key[h[r]] : key[r];
#pragma unroll
                        for (int r = 0; r < kGroupItems; ++r) {
                            if (!((pend >> r) & 1u)) continue;
                            if (cur[r] == key[r])
                                found |= 1u << r;
                            else
                                h[r] = (h[r] + 1u) & (uint32_t)(kSlots - 1);
                        }
                        pend &= ~found;
                    }
                    if (pend != 0u) raise_internal(ctl, kSiteGroupLookup);
#pragma unroll
                    for (int r = 0; r < kGroupItems; ++r)
                        slot[r] = (found >> r) & 1u ? h[r] : kEmptyKey;
                }
                uint32_t mask = 0u, cnt = 0u;
#pragma unroll
                for (int r = 0; r < kGroupItems; ++r) {
                    if (slot[r] != kEmptyKey && (s_cnt[slot[r]] & kRepFlag)) {
                        mask |= 1u << r;
                        ++cnt;
                    }
                }
                uint32_t chunk_rep;
                const uint32_t k0 = block_excl(cnt, s_tmp[5], &chunk_rep);  // synchronises
                {
                    uint32_t k = k0;
#pragma unroll
                    for (int r = 0; r < kGroupItems; ++r)
                        if (mask & (1u << r)) s_rep[k++] = slot[r];
                }
                __syncthreads();
                if (wave == 0) {
                    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
                    for (uint32_t j0 = 0; j0 < chunk_rep; j0 += 64) {
                        const uint32_t j = j0 + (uint32_t)lane;
                        const bool act = j < chunk_rep;
                        const uint32_t sl = act ? s_rep[j] : 0u;
                        const uint64_t peers = match_peers(sl, TB, __ballot(act));
                        const uint32_t before = (uint32_t)__popcll(peers & lt_mask);
                        const int ld = __ffsll((long long)peers) - 1;
                        const int leader = ld < 0 ? 0 : ld;
                        uint32_t st = 0u;
                        if (act && before == 0u) {
                            st = s_cnt[sl];
                            s_cnt[sl] = st + (uint32_t)__popcll(peers);
                        }
                        st = __shfl(st, leader, 64);
                        if (act) s_rep[j] = (st & ~kRepFlag) + before;
                    }
                }
                __syncthreads();
                uint32_t k = k0;
#pragma unroll
                for (int r = 0; r < kGroupItems; ++r) {
                    if (mask & (1u << r)) {
                        const uint32_t pos = s_rep[k++];
                        if ((int64_t)pos >= s0 && (int64_t)pos < s0 + (int64_t)n &&
                            (int64_t)val[r] < m)
                            info[val[r]] = (int32_t)pos;
                        else
                            raise_internal(ctl, kSiteGroupPlace);
                    }
                }
                __syncthreads();  // s_rep is reused by the next chunk
            }
        }
        rep_base += t_rep;

        // ---- next range, depth first ----
        while (level > 0 && (ridx & 1u)) {
            --level;
            ridx >>= 1;
        }
        if (level == 0) break;
        ridx += 1u;
        if (level < depth) {  // the sibling is split as far as this one was
            ridx <<= (depth - level);
            level = depth;
        }
        __syncthreads();  // the table is cleared for the next range
    }
    __syncthreads();
    if (tid < 3) wstats[b * 3 + tid] = s_stat[tid];
    }
}

int group_table_bits(int64_t m, int bins) {
    const int64_t mean = bins > 0 ? (m + bins - 1) / bins : m;
    int tb = kTableBitsMin;
    while (tb < kTableBitsMax && mean > ((int64_t)1 << tb) / 4 * 3) ++tb;
    return tb;
}

hipError_t launch_group(Control* ctl, const uint32_t* keys, const uint32_t* vals, int64_t m,
                        int64_t N, const uint32_t* hist, const uint32_t* bstart, int32_t* info,
                        uint4* shorts, uint4* pieces, uint4* combs, ListCaps caps,
                        uint32_t* wstats, int bins, int key_bits, int grid_cap,
                        int table_bits, hipStream_t s) {
    if (m == 0) return hipSuccess;
    if (bins < 2 || bins > kMaxBins || (bins & (bins - 1)) != 0) return hipErrorInvalidValue;
    const int shift = __builtin_ctz((unsigned)bins);
    const int sub_bits = key_bits > shift ? key_bits - shift : 0;
    // the bitmap path unless a table size is asked for
    const bool bm = table_bits == 0 && sub_bits <= kBitmapBits;
    if (table_bits == 0) table_bits = bm ? kTableBitsMin : group_table_bits(m, bins);
    const int grid = grid_cap > 0 && grid_cap < bins ? grid_cap : bins;
#define HUGE_GROUP_LAUNCH(TB, BM)                                                             \
    hipLaunchKernelGGL((k_group<TB, BM>), dim3((unsigned)grid), dim3(kBlock), 0, s, ctl, keys, \
                       vals, m, N, hist, bstart, info, shorts, pieces, combs, caps, wstats,    \
                       bins, shift, sub_bits)
    if (bm) {
        HUGE_GROUP_LAUNCH(kTableBitsMin, true);
    } else {
        switch (table_bits) {
            case 12: HUGE_GROUP_LAUNCH(12, false); break;
            case 13: HUGE_GROUP_LAUNCH(13, false); break;
            case 14: HUGE_GROUP_LAUNCH(14, false); break;
            default: return hipErrorInvalidValue;
        }
    }
#undef HUGE_GROUP_LAUNCH
    return hipGetLastError();
}

}  // namespace huge
