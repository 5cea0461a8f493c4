// Grouping of the rows a batch touches (the de-duplication of HUGE Sec. 3.3.2):
// which rows occur once -- those are updated in place by the step -- and, for
// every row that occurs several times, the list of its occurrences in
// occurrence order, which is the order in which its contributions are summed.
//
// Occurrence o = i (2 + K) + slot of positive i carries key N + src (slot 0,
// source table) or the context row id (destination, negatives).
//   1. the occurrences of each digit (lowest 8-10 key bits) per tile -- for
//      the step, counted by the sampler as it writes the keys, a tile being
//      one sampler workgroup's keys (at most kSortTile); elsewhere by
//      k_tile_count over tiles of kSortTile -- then k_tile_scan: their sums
//      over earlier tiles, and the bucket sizes;
//   2. k_radix_pass: one stable scatter of the occurrences into bucket
//      (digit) order, each bucket in occurrence order; no tile waits for
//      another;
//   3. k_group: one workgroup per bucket finds the bucket's repeated keys,
//      gives every repeated row a contiguous range of duplicate-buffer slots
//      (inside the bucket's own range of positions), writes the slot of each
//      of its occurrences, in occurrence order, to info[o], and lists the
//      repeated rows for the finish kernel.
// All of them run beside the previous batch's fused step: 256-thread
// workgroups whose waves hold few registers (one item per thread at a time,
// loads issued in small groups) and work mostly in LDS.
#include "common.hpp"
#include "device.hpp"

namespace huge {

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

__device__ __forceinline__ uint64_t lanes_below() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// ---------------------------------------------------------------------------
// Digit counts of tile t (kSortTile consecutive keys, coalesced reads in
// groups of four per thread): tcount[t * bins + d], digit d = bits
// [shift, shift + bits) of the key.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) HUGE_BESIDE void k_tile_count(const Control* __restrict__ ctl,
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
        for (int r0 = 0; r0 < kPer; r0 += 4) {
            uint32_t k[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t o = base + (int64_t)(r0 + j) * kBlock + threadIdx.x;
                k[j] = o < m ? keys[o] : 0xFFFFFFFFu;
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t o = base + (int64_t)(r0 + j) * kBlock + threadIdx.x;
                if (o < m) atomicAdd(&s_cnt[(k[j] >> shift) & (uint32_t)(bins - 1)], 1u);
            }
        }
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
// kScanDigits digits; its kBlock / kScanDigits thread groups each sum a
// contiguous range of tiles, and the ranges are combined through LDS.
// ---------------------------------------------------------------------------
constexpr int kScanGroups = kBlock / kScanDigits;

__global__ __launch_bounds__(kBlock) HUGE_BESIDE void k_tile_scan(const Control* __restrict__ ctl,
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
#pragma unroll 4
    for (int64_t t = t0; t < t1; ++t) sum += tcount[t * bins + d];
    s_part[g][dl] = sum;
    __syncthreads();
    uint32_t run = 0, total = 0;
#pragma unroll 8
    for (int h = 0; h < kScanGroups; ++h) {
        const uint32_t v = s_part[h][dl];
        run += h < g ? v : 0u;
        total += v;
    }
    if (g == 0) hist[d] = total;
#pragma unroll 1
    for (int64_t t = t0; t < t1; ++t) {
        const uint32_t v = tcount[t * bins + d];
        tprefix[t * bins + d] = run;
        run += v;
    }
}

hipError_t launch_tile_scan(Control* ctl, const uint32_t* tcount, int64_t m, int64_t tile,
                            int bits, uint32_t* tprefix, uint32_t* hist, hipStream_t s) {
    if (tile < 1 || tile > kSortTile) return hipErrorInvalidValue;
    const int64_t tiles = (m + tile - 1) / tile;
    if (tiles == 0) return hipSuccess;
    if (bits < kMinDigitBits || bits > kMaxDigitBits) return hipErrorInvalidValue;
    static_assert((1 << kMinDigitBits) % kScanDigits == 0, "whole digit groups");
    hipLaunchKernelGGL(k_tile_scan, dim3((unsigned)((1 << bits) / kScanDigits)), dim3(kBlock), 0,
                       s, ctl, tcount, tiles, bits, tprefix, hist);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Stable scatter by BITS bits at `shift` over a tile of tile_keys <=
// kSortTile consecutive items; wave w owns the w-th quarter of the tile's
// items, in rounds of 64.
//   count: lanes of a round holding the same digit are found with BITS
//          ballots; the lowest of them adds the round's count to the wave's
//          LDS counter of that digit (one writer per digit and round);
//   order: per digit (kBins / kBlock digits per thread) the tile-local start,
//          the wave offsets, and the shift to the global position: bucket
//          start + the digit's count in earlier tiles - tile-local start;
//   place: the rounds again; a lane's position is its wave's running offset
//          of the digit plus the lanes of its round before it; the items go
//          to LDS in digit order (stable);
//   write: LDS position p goes to global position p + shift of its digit:
//          runs of equal digits are contiguous, so the writes coalesce.
// vals_out (if not null) receives the position of each key in keys_in;
// bstart (if not null) the first position of each bucket.
// ---------------------------------------------------------------------------
template <int BITS>
__global__ __launch_bounds__(kBlock) HUGE_BESIDE void k_radix_pass(
    Control* __restrict__ ctl, const uint32_t* __restrict__ keys_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t m,
    int64_t tile_keys, int shift, const uint32_t* __restrict__ hist,
    const uint32_t* __restrict__ tprefix, uint32_t* __restrict__ bstart) {
    constexpr int kBins = 1 << BITS;
    constexpr int kWaves = kBlock / 64;
    constexpr int kDpt = kBins / kBlock;  // digits per thread
    static_assert(kDpt >= 1 && kBins % kBlock == 0, "whole digits per thread");
    // dynamic LDS (radix_lds_bytes<BITS>()): with a static size this large
    // the compiler, seeing one wave per SIMD at most, would not keep to the
    // HUGE_BESIDE register budget
    extern __shared__ uint32_t s_dyn[];
    uint32_t(*const s_wave)[kBins] = reinterpret_cast<uint32_t(*)[kBins]>(s_dyn);
    int32_t* const s_delta = reinterpret_cast<int32_t*>(s_dyn + kWaves * kBins);
    uint32_t* const s_in = s_dyn + (kWaves + 1) * kBins;  // the tile's keys in input order
    uint32_t* const s_keys = s_in + kSortTile;            // ... in digit order
    uint32_t* const s_vals = s_keys + kSortTile;          // and their input positions
    __shared__ uint32_t s_tmp[2][kWaves];

    if (ctl->step_bad) return;  // uniform: the call is a no-op

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int64_t tile = blockIdx.x;
    const int64_t tile_base = tile * tile_keys;  // tile_keys <= kSortTile
    const int64_t valid_n = (m - tile_base) < tile_keys ? (m - tile_base) : tile_keys;
    // wave w owns the w-th quarter of the tile (a multiple of 64 items), in
    // order, so the scatter stays stable
    const int rounds = (int)((valid_n + kWaves * 64 - 1) / (kWaves * 64));
    const int wbase = wave * rounds * 64;

    for (int j = tid; j < kWaves * kBins; j += kBlock) (&s_wave[0][0])[j] = 0u;
    for (int p = tid; p < valid_n; p += kBlock) s_in[p] = keys_in[tile_base + p];
    __syncthreads();

    // count
    for (int r = 0; r < rounds; ++r) {
        const int p = wbase + r * 64 + lane;
        const bool valid = p < valid_n;
        const uint32_t dg = valid ? (s_in[p] >> shift) & (kBins - 1) : 0u;
        const uint64_t peers = match_peers(dg, BITS, __ballot(valid));
        if (valid && (peers & lanes_below()) == 0)
            s_wave[wave][dg] += (uint32_t)__popcll(peers);
    }
    __syncthreads();

    // order
    uint32_t cnt_sum = 0, hist_sum = 0;
#pragma unroll
    for (int j = 0; j < kDpt; ++j) {
        const int d = tid * kDpt + j;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) cnt_sum += s_wave[w][d];
        hist_sum += hist[d];
    }
    uint32_t total;
    uint32_t local = block_excl(cnt_sum, s_tmp[0], &total);
    uint32_t gstart = block_excl(hist_sum, s_tmp[1], &total);
#pragma unroll
    for (int j = 0; j < kDpt; ++j) {
        const int d = tid * kDpt + j;
        uint32_t run = local;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const uint32_t c = s_wave[w][d];
            s_wave[w][d] = run;
            run += c;
        }
        s_delta[d] = (int32_t)(gstart + tprefix[tile * kBins + d]) - (int32_t)local;
        if (bstart != nullptr && tile == 0) bstart[d] = gstart;
        gstart += hist[d];
        local = run;
    }
    __syncthreads();

    // place
    for (int r = 0; r < rounds; ++r) {
        const int p = wbase + r * 64 + lane;
        const bool valid = p < valid_n;
        const uint32_t key = valid ? s_in[p] : 0u;
        const uint32_t dg = (key >> shift) & (kBins - 1);
        const uint64_t peers = match_peers(dg, BITS, __ballot(valid));
        const uint32_t before = (uint32_t)__popcll(peers & lanes_below());
        uint32_t off = 0;
        if (valid) off = s_wave[wave][dg];  // every lane reads before the first lane adds
        if (valid && before == 0) s_wave[wave][dg] = off + (uint32_t)__popcll(peers);
        if (valid && off + before < (uint32_t)kSortTile) {
            s_keys[off + before] = key;
            s_vals[off + before] = (uint32_t)(tile_base + p);
        } else if (valid) {
            raise_internal(ctl, kSiteRadixDest);
        }
    }
    __syncthreads();

    // write
    for (int p = tid; p < valid_n; p += kBlock) {
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

// Dynamic LDS bytes of k_radix_pass<BITS>.
template <int BITS>
constexpr size_t radix_lds_bytes() {
    return sizeof(uint32_t) * ((size_t)(kBlock / 64 + 1) * (1 << BITS) + 3 * (size_t)kSortTile);
}

template <int BITS>
hipError_t launch_radix_bits(Control* ctl, const uint32_t* keys_in, uint32_t* keys_out,
                             uint32_t* vals_out, int64_t m, int64_t tile, int shift,
                             const uint32_t* hist, const uint32_t* tprefix, uint32_t* bstart,
                             int64_t tiles, hipStream_t s) {
    // LDS beyond 64 KB is asked for explicitly, once per variant
    static bool lds_set = false;
    if (!lds_set) {
        const hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&k_radix_pass<BITS>),
            hipFuncAttributeMaxDynamicSharedMemorySize, (int)radix_lds_bytes<BITS>());
        if (e != hipSuccess) return e;
        lds_set = true;
    }
    hipLaunchKernelGGL(k_radix_pass<BITS>, dim3((unsigned)tiles), dim3(kBlock),
                       radix_lds_bytes<BITS>(), s, ctl, keys_in, keys_out, vals_out, m, tile,
                       shift, hist, tprefix, bstart);
    return hipGetLastError();
}

hipError_t launch_radix_pass(Control* ctl, const uint32_t* keys_in, uint32_t* keys_out,
                             uint32_t* vals_out, int64_t m, int64_t tile, int bits, int shift,
                             const uint32_t* hist, const uint32_t* tprefix, uint32_t* bstart,
                             hipStream_t s) {
    if (tile < 1 || tile > kSortTile) return hipErrorInvalidValue;
    const int64_t tiles = (m + tile - 1) / tile;
    if (tiles == 0) return hipSuccess;
    if (shift < 0 || shift > 31) return hipErrorInvalidValue;
#define HUGE_RADIX_LAUNCH(B)                                                                  \
    return launch_radix_bits<B>(ctl, keys_in, keys_out, vals_out, m, tile, shift, hist,       \
                                tprefix, bstart, tiles, s)
    switch (bits) {
        case 8: HUGE_RADIX_LAUNCH(8);
        case 9: HUGE_RADIX_LAUNCH(9);
        case 10: HUGE_RADIX_LAUNCH(10);
        default: return hipErrorInvalidValue;
    }
#undef HUGE_RADIX_LAUNCH
}

// ---------------------------------------------------------------------------
// Grouping of one bucket (its items are in occurrence order).
//
// A first pass copies the bucket's keys (up to kGroupCacheKeys) and
// occurrence indices (up to kGroupCacheVals) to LDS, in one round of loads.
// With BM (the bucket's keys differ in at most kBitmapBits bits above the
// bucket digit) the same pass sets, per item, the key's bit in an LDS bitmap
// and, where it was set already, the key's bit in a second bitmap of
// repeated keys; it also counts the bucket's distinct source and destination
// rows.  Only keys marked repeated take part in what follows.
//
// The (repeated) keys are counted in an LDS hash table of kGroupSlots slots
// (linear probing).  A bucket with more than 3/4 of the slots in distinct
// keys is split into key ranges by further hash bits, each range counted and
// placed in turn (depth first over the binary tree of ranges); at depth 32 a
// range holds one key value, so the split ends.  A count that overflows
// stops at the first chunk that would load the table past 7/8, and the
// number of distinct keys seen so far, scaled to the whole bucket, sets how
// many levels the split descends at once (later sibling ranges start at
// that depth).  Per range:
//   count:  every item of the range inserts its key and counts it;
//   emit:   rows counted more than once get consecutive duplicate-buffer
//           slots (positions of the bucket, after those of earlier ranges),
//           and a work record: a short run or a piece appended to the
//           batch's lists, or pieces plus a combine record (in the bucket's
//           own region) for a run longer than kPiece;
//   place:  the repeated items, taken in occurrence order (chunk by chunk,
//           compacted, then ranked by one wave 64 at a time), receive their
//           row's next slot: info[o] = slot.
// At the end the bucket's record counts go to bcount[b].  No step waits for
// another workgroup; the only device-scope atomics reserve a range's places
// in the batch's record lists.  Where a row's range lands
// depends on the order of the hash insertions, the order of its occurrences
// does not: every sum is taken in occurrence order.  Items that occur once
// keep info = -1.
// ---------------------------------------------------------------------------
constexpr uint32_t kEmptyKey = 0xFFFFFFFFu;   // keys are below 2N <= 2^32 - 2
constexpr uint32_t kRepFlag = 0x80000000u;    // table count word: a repeated row, next slot
constexpr int kMaxProbe = 512;                // a longer probe also splits the range

// Slot of a key in a table of 2^tbits slots.
__device__ __forceinline__ uint32_t slot_hash(uint32_t key, int tbits) {
    return (key * 0x85EBCA6Bu) >> (32 - tbits);
}

__device__ __forceinline__ bool in_range(uint32_t key, int level, uint32_t idx) {
    return level == 0 || ((key * 0xC2B2AE35u) >> (32 - level)) == idx;
}

// Dynamic LDS words of k_group<BM>.
template <bool BM>
constexpr size_t group_lds_words() {
    return 2 * kGroupSlots + kGroupCacheKeys + kGroupCacheVals + kGroupChunk +
           (BM ? 2 * ((1 << kBitmapBits) / 32) : 0);
}

template <bool BM>
__global__ __launch_bounds__(kBlock) HUGE_BESIDE_72 void k_group(
    Control* __restrict__ ctl, const uint32_t* __restrict__ keys,
    const uint32_t* __restrict__ vals, int64_t m, int64_t N, const uint32_t* __restrict__ hist,
    const uint32_t* __restrict__ bstart, int32_t* __restrict__ info, uint4* __restrict__ shorts,
    uint4* __restrict__ pieces, uint4* __restrict__ combs, uint32_t* __restrict__ ccount,
    uint4* __restrict__ bcount, ListCaps caps, uint32_t* __restrict__ wstats, int bins, int shift,
    int sub_bits) {
    constexpr int kBitWords = (1 << kBitmapBits) / 32;           // words of one bitmap
    // The large arrays live in dynamic LDS (group_lds_words<BM>() words): the
    // compiler then keeps to the HUGE_BESIDE register budget, which a static
    // size above a fifth of the LDS would let it exceed.
    extern __shared__ uint32_t s_dyn[];
    uint32_t* const s_key = s_dyn;                          // [kGroupSlots]
    uint32_t* const s_cnt = s_key + kGroupSlots;            // count; after emit, kRepFlag | next slot
    uint32_t* const s_ckey = s_cnt + kGroupSlots;           // [kGroupCacheKeys]
    uint32_t* const s_cval = s_ckey + kGroupCacheKeys;      // [kGroupCacheVals]
    // repeated items of a chunk in order: their table slot, then their
    // duplicate-buffer slot
    uint32_t* const s_rep = s_cval + kGroupCacheVals;       // [kGroupChunk]
    uint32_t* const s_seen = s_rep + kGroupChunk;           // [kBitWords] with BM
    uint32_t* const s_dup = s_seen + kBitWords;             // [kBitWords] with BM
    __shared__ uint32_t s_tmp[6][kBlock / 64];
    __shared__ uint32_t s_distinct, s_fail, s_nrep;
    __shared__ uint32_t s_stat[3];
    __shared__ uint32_t s_rbase[2];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // the first failed internal check of this thread, raised once at the end
    // (one atomic site keeps its operands out of the registers of the loops)
    uint32_t bad = 0u;
#define HUGE_FAIL(site) (bad = bad ? bad : (uint32_t)(site))
    for (int b = blockIdx.x; b < bins; b += gridDim.x) {
    __syncthreads();  // LDS of the previous bucket
    if (tid < 3) s_stat[tid] = 0u;
    if (tid == 0) s_nrep = 0u;
    const uint32_t n = ctl->step_bad ? 0u : hist[b];
    const int64_t s0 = n ? (int64_t)bstart[b] : 0;
    if (n == 0u || s0 + (int64_t)n > m) {
        if (n != 0u && tid == 0) HUGE_FAIL(kSiteGroupBucket);
        if (tid < 3) wstats[b * 3 + tid] = 0u;
        if (tid == 0) bcount[b] = make_uint4(0u, 0u, 0u, 0u);
        continue;
    }
    const bool keys_cached = n <= (uint32_t)kGroupCacheKeys;
    const bool vals_cached = n <= (uint32_t)kGroupCacheVals;
    // the kGroupItems keys of this thread in chunk c0
    // (after the compaction: of the first nw items)
    auto load_keys = [&](uint32_t c0, uint32_t nlim, uint32_t (&k)[kGroupItems]) {
        const uint32_t e0 = c0 + (uint32_t)(tid * kGroupItems);
        if (keys_cached) {
#pragma unroll
            for (int r = 0; r < kGroupItems; ++r) k[r] = e0 + r < nlim ? s_ckey[e0 + r] : 0u;
        } else {
            const uint32_t* kp = keys + s0 + e0;
#pragma unroll
            for (int r = 0; r < kGroupItems; ++r) k[r] = e0 + r < nlim ? kp[r] : 0u;
        }
    };

    // ---- copy to LDS; repeated keys (BM) ----
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
    }
    if (keys_cached || vals_cached) {  // coalesced: item j + q kBlock by thread j
        for (uint32_t e0 = 0; e0 < n; e0 += 4 * kBlock) {
            uint32_t kk[4], vv[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t e = e0 + (uint32_t)(q * kBlock + tid);
                kk[q] = e < n && keys_cached ? keys[s0 + e] : 0u;
                vv[q] = e < n && vals_cached ? vals[s0 + e] : 0u;
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t e = e0 + (uint32_t)(q * kBlock + tid);
                if (e < n && keys_cached) s_ckey[e] = kk[q];
                if (e < n && vals_cached) s_cval[e] = vv[q];
            }
        }
    }
    __syncthreads();
    if (BM) {
        uint32_t nS = 0, nT = 0, nR = 0;
        for (uint32_t c0 = 0; c0 < n; c0 += kGroupChunk) {
            uint32_t k[kGroupItems];
            load_keys(c0, n, k);
#pragma unroll 1
            for (int r = 0; r < kGroupItems; ++r) {
                const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                if (e >= n) continue;
                const uint32_t sub = k[r] >> shift, w = sub >> 5, bit = 1u << (sub & 31u);
                if (w >= bit_words) {
                    HUGE_FAIL(kSiteGroupBits);
                    continue;
                }
                const uint32_t old = atomicOr(&s_seen[w], bit);
                if (old & bit) {
                    atomicOr(&s_dup[w], bit);
                    ++nR;
                } else if ((int64_t)k[r] >= N) {
                    ++nS;
                } else {
                    ++nT;
                }
            }
        }
        if (nS) atomicAdd(&s_stat[0], nS);
        if (nT) atomicAdd(&s_stat[1], nT);
        if (nR) atomicAdd(&s_nrep, nR);
        __syncthreads();
    }
    // with the bitmap: nothing repeated, nothing to group
    const bool any = !BM || s_nrep != 0u;

    // With the bitmap and the whole bucket in LDS, only the items of
    // repeated keys are grouped: they are compacted to the front of the LDS
    // copy, in occurrence order (chunk by chunk; an item moves only to a
    // lower position, so no item is overwritten before it is read), and
    // the hash table is sized to them.
    uint32_t nw = n;  // items the count and the placement go through
    int tbits = kGroupTableBits;
    if (BM && any && keys_cached && vals_cached) {
        uint32_t out = 0;
        for (uint32_t c0 = 0; c0 < n; c0 += kGroupChunk) {
            uint32_t kk[kGroupItems], vv[kGroupItems];
            uint32_t mask = 0u, cnt = 0u;
            const uint32_t e0 = c0 + (uint32_t)(tid * kGroupItems);
#pragma unroll
            for (int r = 0; r < kGroupItems; ++r) {
                kk[r] = e0 + r < n ? s_ckey[e0 + r] : 0u;
                vv[r] = e0 + r < n ? s_cval[e0 + r] : 0u;
            }
#pragma unroll 1
            for (int r = 0; r < kGroupItems; ++r) {
                if (e0 + r < n && repeated(kk[r])) {
                    mask |= 1u << r;
                    ++cnt;
                }
            }
            uint32_t total;
            uint32_t p = out + block_excl(cnt, s_tmp[0], &total);  // synchronises
#pragma unroll 1
            for (int r = 0; r < kGroupItems; ++r) {
                if (mask & (1u << r)) {
                    s_ckey[p] = kk[r];
                    s_cval[p] = vv[r];
                    ++p;
                }
            }
            out += total;
            __syncthreads();  // s_tmp is reused
        }
        nw = out;
        tbits = 6;
        while (tbits < kGroupTableBits && (1u << tbits) < 2u * nw) ++tbits;
    }
    const uint32_t tsize = 1u << tbits;
    const uint32_t tmask = tsize - 1u;
    const uint32_t tmax = tsize / 4u * 3u;   // distinct keys a range may hold
    const uint32_t tload = tsize / 8u * 7u;  // table load a count stays below

    // the bucket's record bounds and regions, and how many records it has written
    const uint32_t c_short = (uint32_t)(n / kShortDiv), c_piece = (uint32_t)(n / kPieceDiv);
    const uint32_t r_comb = (uint32_t)(s0 / kCombDiv), c_comb = (uint32_t)(n / kCombDiv);
    const uint32_t r_part = (uint32_t)(s0 / kPartDiv), c_part = (uint32_t)(n / kPartDiv);
    uint32_t nb_short = 0, nb_piece = 0, nb_comb = 0, nb_part = 0;

    uint32_t rep_base = 0;  // slots handed out to earlier ranges
    int level = 0, depth = 0;  // depth: where the next sibling range starts
    uint32_t ridx = 0;
    auto lookup = [&](uint32_t key) -> uint32_t {
        uint32_t h = slot_hash(key, tbits);
        for (int probe = 0; probe < kMaxProbe; ++probe) {
            const uint32_t kk = s_key[h];
            if (kk == key) return h;
            if (kk == kEmptyKey) return kEmptyKey;
            h = (h + 1u) & tmask;
        }
        return kEmptyKey;
    };
    while (any) {
        // ---- count ----
#pragma unroll 1
        for (uint32_t q = tid; q < tsize; q += kBlock) {
            s_key[q] = kEmptyKey;
            s_cnt[q] = 0u;
        }
        if (tid == 0) {
            s_distinct = 0u;
            s_fail = 0u;
        }
        __syncthreads();
        uint32_t seen = 0;  // items the count went through
        bool over = false;
        for (uint32_t c0 = 0; c0 < nw; c0 += kGroupChunk) {
            const uint32_t len = nw - c0 < (uint32_t)kGroupChunk ? nw - c0 : (uint32_t)kGroupChunk;
            if (s_distinct + len > tload) {  // uniform: the table could fill up
                over = true;
                break;
            }
            uint32_t k[kGroupItems];
            load_keys(c0, nw, k);
            uint32_t fresh = 0u;
#pragma unroll 1
            for (int r = 0; r < kGroupItems; ++r) {
                const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                if (e >= nw || !in_range(k[r], level, ridx) || !repeated(k[r])) continue;
                uint32_t h = slot_hash(k[r], tbits);
                bool found = false;
                for (int probe = 0; probe < kMaxProbe; ++probe) {
                    const uint32_t old = atomicCAS(&s_key[h], kEmptyKey, k[r]);
                    if (old == kEmptyKey || old == k[r]) {
                        fresh += old == kEmptyKey ? 1u : 0u;
                        atomicAdd(&s_cnt[h], 1u);
                        found = true;
                        break;
                    }
                    h = (h + 1u) & tmask;
                }
                if (!found) s_fail = 1u;
            }
            if (fresh) atomicAdd(&s_distinct, fresh);
            __syncthreads();
            seen = c0 + len;
            if (s_fail || s_distinct > tmax) {  // uniform
                over = true;
                break;
            }
        }
        if (over) {
            // split the range; its first part next (uniform)
            int add = 1;
            if (!s_fail && seen > 0u) {
                const uint64_t est = (uint64_t)s_distinct * nw / seen;
                while (add < 8 && est > ((uint64_t)tmax << add) / 4u * 3u) ++add;
            }
            __syncthreads();
            if (level >= 32) {  // cannot happen: a depth-32 range holds one key value
                HUGE_FAIL(kSiteGroupDepth);
                goto finished;
            }
            if (add > 32 - level) add = 32 - level;
            level += add;
            ridx <<= add;
            if (depth < level) depth = level;
            continue;
        }

        {
        // ---- emit ----
        // this thread's table slots (tid, tid + kBlock, ...; conflict-free
        // LDS reads): statistics, slot counts, record counts; slots and
        // records are handed out thread by thread
        uint32_t nS = 0, nT = 0, nrep = 0, nshort = 0, npiece = 0, ncomb = 0, npart = 0;
#pragma unroll 1
        for (uint32_t q = tid; q < tsize; q += kBlock) {
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
        const uint32_t x_rep = block_excl(nrep, s_tmp[0], &t_rep);
        const uint32_t x_short = block_excl(nshort, s_tmp[1], &t_short);
        const uint32_t x_piece = block_excl(npiece, s_tmp[2], &t_piece);
        const uint32_t x_comb = block_excl(ncomb, s_tmp[3], &t_comb);
        const uint32_t x_part = block_excl(npart, s_tmp[4], &t_part);
        if (nS) atomicAdd(&s_stat[0], nS);
        if (nT) atomicAdd(&s_stat[1], nT);
        // the range's short runs and pieces are appended to the batch's lists
        // at positions reserved by one device-scope atomic each (the finish
        // kernel takes each record alone, so their order is free)
        if (tid == 0) {
            s_rbase[0] = t_short ? atomicAdd(&ctl->nshort, t_short) : 0u;
            s_rbase[1] = t_piece ? atomicAdd(&ctl->npiece, t_piece) : 0u;
        }
        __syncthreads();
        const uint32_t b_short = s_rbase[0], b_piece = s_rbase[1];
        // uniform: every thread has the same totals and bases
        const bool fits = (uint64_t)nb_short + t_short <= c_short &&
                          (uint64_t)nb_piece + t_piece <= c_piece &&
                          (uint64_t)nb_comb + t_comb <= c_comb &&
                          (uint64_t)nb_part + t_part <= c_part &&
                          (uint64_t)rep_base + t_rep <= n &&
                          (uint64_t)b_short + t_short <= caps.shorts &&
                          (uint64_t)b_piece + t_piece <= caps.pieces &&
                          (uint64_t)r_comb + c_comb <= caps.combs &&
                          (uint64_t)r_part + c_part <= caps.parts;
        if (!fits) {  // cannot happen: the regions bound every bucket
            HUGE_FAIL(kSiteGroupLists);
            goto finished;
        }
        {
            uint32_t pos = (uint32_t)s0 + rep_base + x_rep;
            uint32_t is = b_short + x_short, ip = b_piece + x_piece;
            uint32_t ic = r_comb + nb_comb + x_comb, ia = r_part + nb_part + x_part;
#pragma unroll 1
            for (uint32_t q = tid; q < tsize; q += kBlock) {
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
                        pieces[ip++] = make_uint4(pos + z * kPiece, len, k, ic + 1u);
                    }
                    combs[ic] = make_uint4(k, ia, np, pos);
                    ccount[ic] = 0u;
                    ++ic;
                    ia += np;
                }
                s_cnt[q] = kRepFlag | pos;
                pos += c;
            }
        }
        nb_short += t_short;
        nb_piece += t_piece;
        nb_comb += t_comb;
        nb_part += t_part;
        if (tid == 0) s_stat[2] += t_rep;
        __syncthreads();

        // ---- place ----
        if (t_rep > 0u) {
            for (uint32_t c0 = 0; c0 < nw; c0 += kGroupChunk) {
                uint32_t k[kGroupItems];
                load_keys(c0, nw, k);
                uint32_t mask = 0u, cnt = 0u;
#pragma unroll 1
                for (int r = 0; r < kGroupItems; ++r) {
                    const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                    if (e >= nw || !in_range(k[r], level, ridx) || !repeated(k[r])) continue;
                    const uint32_t h = lookup(k[r]);
                    if (h == kEmptyKey) {
                        HUGE_FAIL(kSiteGroupLookup);
                        continue;
                    }
                    if (s_cnt[h] & kRepFlag) {
                        mask |= 1u << r;
                        ++cnt;
                    }
                }
                uint32_t chunk_rep;
                const uint32_t k0 = block_excl(cnt, s_tmp[5], &chunk_rep);  // synchronises
                {
                    uint32_t kk = k0;
#pragma unroll 1
                    for (int r = 0; r < kGroupItems; ++r)
                        if (mask & (1u << r)) s_rep[kk++] = lookup(k[r]);
                }
                __syncthreads();
                if (wave == 0) {
                    for (uint32_t j0 = 0; j0 < chunk_rep; j0 += 64) {
                        const uint32_t j = j0 + (uint32_t)lane;
                        const bool act = j < chunk_rep;
                        const uint32_t sl = act ? s_rep[j] : 0u;
                        const uint64_t peers = match_peers(sl, tbits, __ballot(act));
                        const uint32_t before = (uint32_t)__popcll(peers & lanes_below());
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
                uint32_t kk = k0;
#pragma unroll 1
                for (int r = 0; r < kGroupItems; ++r) {
                    if (mask & (1u << r)) {
                        const uint32_t pos = s_rep[kk++];
                        const uint32_t e = c0 + (uint32_t)(tid * kGroupItems + r);
                        const uint32_t o = vals_cached ? s_cval[e] : vals[s0 + e];
                        if ((int64_t)pos >= s0 && (int64_t)pos < s0 + (int64_t)n && (int64_t)o < m)
                            info[o] = (int32_t)pos;
                        else
                            HUGE_FAIL(kSiteGroupPlace);
                    }
                }
                __syncthreads();  // s_rep is reused by the next chunk
            }
        }
        rep_base += t_rep;
        }

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
    if (tid == 0) bcount[b] = make_uint4(nb_short, nb_piece, nb_comb, 0u);
    }
finished:
    if (bad) raise_internal(ctl, bad);
#undef HUGE_FAIL
}

hipError_t launch_group(Control* ctl, const uint32_t* keys, const uint32_t* vals, int64_t m,
                        int64_t N, const uint32_t* hist, const uint32_t* bstart, int32_t* info,
                        uint4* shorts, uint4* pieces, uint4* combs, uint32_t* ccount,
                        uint4* bcount, ListCaps caps, uint32_t* wstats, int bins, int key_bits,
                        hipEvent_t stop, bool* launched, hipStream_t s) {
    *launched = false;
    if (m == 0) return hipSuccess;
    if (bins < 2 || bins > kMaxBins || (bins & (bins - 1)) != 0) return hipErrorInvalidValue;
    const int shift = __builtin_ctz((unsigned)bins);
    const int sub_bits = key_bits > shift ? key_bits - shift : 0;
    // LDS beyond 64 KB is asked for explicitly, once per variant
    static bool lds_set[2] = {false, false};
    const bool bm = sub_bits <= kBitmapBits;
    if (!lds_set[bm]) {
        const size_t bytes = (bm ? group_lds_words<true>() : group_lds_words<false>()) * 4;
        const void* fn = bm ? reinterpret_cast<const void*>(&k_group<true>)
                            : reinterpret_cast<const void*>(&k_group<false>);
        const hipError_t e =
            hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
        if (e != hipSuccess) return e;
        lds_set[bm] = true;
    }
    if (bm) {
        hipExtLaunchKernelGGL(k_group<true>, dim3((unsigned)bins), dim3(kBlock),
                              group_lds_words<true>() * sizeof(uint32_t), s, nullptr, stop, 0,
                              ctl, keys, vals, m, N, hist, bstart, info, shorts, pieces, combs,
                              ccount, bcount, caps, wstats, bins, shift, sub_bits);
    } else {
        hipExtLaunchKernelGGL(k_group<false>, dim3((unsigned)bins), dim3(kBlock),
                              group_lds_words<false>() * sizeof(uint32_t), s, nullptr, stop, 0,
                              ctl, keys, vals, m, N, hist, bstart, info, shorts, pieces, combs,
                              ccount, bcount, caps, wstats, bins, shift, sub_bits);
    }
    const hipError_t e = hipGetLastError();
    *launched = e == hipSuccess;
    return e;
}

}  // namespace huge
