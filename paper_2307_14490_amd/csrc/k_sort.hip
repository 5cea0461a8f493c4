// Grouping of the rows a batch touches: a stable LSD radix sort of the
// occurrence keys (one kernel per 8-bit digit, single pass over the data with
// decoupled look-back between tiles), then run marking on the sorted keys.
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

// One pass of 8 bits at shift 8 * pass.  Tile = kSortTile consecutive items,
// wave w of the tile owns a quarter of them, in kSortItems rounds of 64.
// Within a round, lanes with the same digit are found with 8 ballots; the
// round's count per digit is added to the wave's LDS counter by one lane,
// whose old value orders the round after the earlier ones.
__global__ __launch_bounds__(kBlock) void k_radix_pass(
    Control* __restrict__ ctl, uint32_t* __restrict__ tickets,
    const uint32_t* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t m, int pass,
    const uint32_t* __restrict__ hist, uint64_t* __restrict__ status, uint32_t tag) {
    __shared__ uint32_t s_wave[4][kRadixBins];
    __shared__ uint32_t s_base[kRadixBins];
    __shared__ uint32_t s_scan[kRadixBins];
    __shared__ uint32_t s_tile;

    if (ctl->step_bad) return;  // uniform: the call is a no-op

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int shift = pass * kRadixBits;

    for (int j = tid; j < 4 * kRadixBins; j += kBlock) (&s_wave[0][0])[j] = 0u;
    if (tid == 0) s_tile = atomicAdd(tickets, 1u);
    // global exclusive prefix of the digit counts (Hillis-Steele in LDS)
    s_scan[tid] = hist[tid];
    __syncthreads();
    for (int off = 1; off < kRadixBins; off <<= 1) {
        const uint32_t add = tid >= off ? s_scan[tid - off] : 0u;
        __syncthreads();
        s_scan[tid] += add;
        __syncthreads();
    }
    const uint32_t global_excl = s_scan[tid] - hist[tid];
    const int64_t tile = s_tile;
    if (tile >= (int64_t)gridDim.x) {  // tickets were not reset: refuse, never wait
        if (tid == 0) raise_error(ctl, kBadInternal);
        return;
    }
    const int64_t base_idx = tile * kSortTile + (int64_t)wave * (kSortTile / 4);

    uint32_t key[kSortItems], val[kSortItems], rank[kSortItems];
    const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t idx = base_idx + r * 64 + lane;
        const bool valid = idx < m;
        key[r] = valid ? keys_in[idx] : 0u;
        val[r] = valid ? (vals_in ? vals_in[idx] : (uint32_t)idx) : 0u;
    }
#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t idx = base_idx + r * 64 + lane;
        const bool valid = idx < m;
        const uint32_t d = (key[r] >> shift) & (kRadixBins - 1);
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < kRadixBits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t ones = __ballot(bit);
            peers &= bit ? ones : ~ones;
        }
        const uint32_t before = (uint32_t)__popcll(peers & lt_mask);
        const int leader = __ffsll((long long)peers) - 1;
        uint32_t old = 0;
        if (valid && before == 0) old = atomicAdd(&s_wave[wave][d], (uint32_t)__popcll(peers));
        old = __shfl(old, leader < 0 ? 0 : leader, 64);
        rank[r] = old + before;
    }
    __syncthreads();

    // Per digit: counts of the four waves -> exclusive offsets; tile count.
    const int d = tid;
    const uint32_t c0 = s_wave[0][d], c1 = s_wave[1][d], c2 = s_wave[2][d], c3 = s_wave[3][d];
    const uint32_t tile_count = c0 + c1 + c2 + c3;
    s_wave[0][d] = 0u;
    s_wave[1][d] = c0;
    s_wave[2][d] = c0 + c1;
    s_wave[3][d] = c0 + c1 + c2;

    // Decoupled look-back over the tiles before this one, for digit d: the
    // words of kLookBatch predecessors are read together, then consumed in
    // order until an inclusive prefix is met.
    uint64_t* my = status + tile * kRadixBins + d;
    uint32_t excl = 0;
    if (tile == 0) {
        lb_store(my, lb_word(tag, kFlagPrefix, tile_count));
    } else {
        lb_store(my, lb_word(tag, kFlagAggregate, tile_count));
        const uint32_t want = tag & 0x3FFFFFFFu;
        int64_t look = tile - 1;
        uint32_t spins = 0;
        bool done = false;
        while (!done) {
            uint64_t w[kLookBatch];
#pragma unroll
            for (int j = 0; j < kLookBatch; ++j)
                w[j] = (look - j >= 0) ? lb_load(status + (look - j) * kRadixBins + d)
                                       : lb_word(want, kFlagPrefix, 0u);
            int used = 0;
#pragma unroll
            for (int j = 0; j < kLookBatch; ++j) {
                if (done || used != j) break;
                const uint64_t flag = (w[j] >> 32) & 3ull;
                if ((uint32_t)(w[j] >> 34) != want || flag == 0ull) break;
                excl += (uint32_t)w[j];
                used = j + 1;
                if (flag == kFlagPrefix) done = true;
            }
            look -= used;
            if (!done && used < kLookBatch) {
                // every earlier tile is resident (it holds a smaller ticket) and
                // publishes without waiting; the bound only guards against a
                // broken invariant, turning it into a reported error
                if (++spins > (1u << 22)) {
                    raise_error(ctl, kBadInternal);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        lb_store(my, lb_word(tag, kFlagPrefix, excl + tile_count));
    }
    s_base[d] = global_excl + excl;
    __syncthreads();

#pragma unroll
    for (int r = 0; r < kSortItems; ++r) {
        const int64_t idx = base_idx + r * 64 + lane;
        if (idx < m) {
            const uint32_t dd = (key[r] >> shift) & (kRadixBins - 1);
            const uint32_t dest = s_base[dd] + s_wave[wave][dd] + rank[r];
            if ((int64_t)dest < m) {
                keys_out[dest] = key[r];
                vals_out[dest] = val[r];
            } else {
                raise_error(ctl, kBadInternal);
            }
        }
    }
}

hipError_t launch_radix_pass(Control* ctl, const uint32_t* keys_in, const uint32_t* vals_in,
                             uint32_t* keys_out, uint32_t* vals_out, int64_t m, int pass,
                             const uint32_t* hist, uint64_t* status, uint32_t tag,
                             hipStream_t s) {
    const int64_t tiles = (m + kSortTile - 1) / kSortTile;
    if (tiles == 0) return hipSuccess;
    hipLaunchKernelGGL(k_radix_pass, dim3((unsigned)tiles), dim3(kBlock), 0, s, ctl,
                       &ctl->tickets[pass], keys_in, vals_in, keys_out, vals_out, m, pass,
                       hist + pass * kRadixBins, status, tag);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Run marking on the sorted keys, one workgroup per window of kChunk sorted
// positions.  Position j (occurrence o = vals[j]):
//   info[o] = -1 if its key occurs once, else j (its slot in the duplicate
//   buffer).  Runs of a repeated key are cut into pieces at window
//   boundaries; each piece becomes a work item {start, len, key, kind} stored
//   in its window's slots work[w * kChunk ..]:
//     kind 0: the whole run -> sum and update the row directly;
//     kind 1: the run's first piece, the run continues past the window ->
//             partial sum to partB[w]; longhead[w] = its start;
//     kind 2: a later piece, starting at the window boundary -> partA[w].
//   A window holds at most one kind-1 piece.  Per window: number of pieces,
//   and {distinct source keys, distinct context keys, repeated occurrences}.
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
    if (ctl->step_bad) return;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if (tid < 3) s_cnt[tid] = 0u;
    if (tid == 0) s_long = 0xFFFFFFFFu;
    __syncthreads();
    const int64_t win = blockIdx.x;
    const int64_t j = win * kChunk + tid;
    bool emit = false, head_S = false, head_T = false, dup = false;
    uint4 rec = make_uint4(0, 0, 0, 0);
    if (j < m) {
        const uint32_t key = keys[j];
        const bool prev_same = j > 0 && keys[j - 1] == key;
        const bool next_same = j + 1 < m && keys[j + 1] == key;
        dup = prev_same || next_same;
        const uint32_t o = vals[j];
        if ((int64_t)o < m) info[o] = dup ? (int32_t)j : -1;
        head_S = !prev_same && (int64_t)key >= N;
        head_T = !prev_same && (int64_t)key < N;
        if (dup && (!prev_same || tid == 0)) {
            const int64_t win_end = (win + 1) * kChunk;
            const int64_t lim = win_end < m ? win_end : m;
            int64_t e = j + 1;
            while (e < lim && keys[e] == key) ++e;
            const bool cont_after = (e == win_end) && (e < m) && keys[e] == key;
            const uint32_t kind = !prev_same ? (cont_after ? 1u : 0u) : 2u;
            rec = make_uint4((uint32_t)j, (uint32_t)(e - j), key, kind);
            emit = true;
            if (kind == 1u) s_long = (uint32_t)j;
        }
    }
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const uint64_t em = __ballot(emit);
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
        wcount[win] = total;
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
