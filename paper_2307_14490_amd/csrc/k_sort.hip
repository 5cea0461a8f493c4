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
// wave w of the tile owns items [w * 1024, (w + 1) * 1024) in 16 rounds of 64.
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

    // Decoupled look-back over the tiles before this one, for digit d.
    uint64_t* my = status + tile * kRadixBins + d;
    uint32_t excl = 0;
    if (tile == 0) {
        lb_store(my, lb_word(tag, kFlagPrefix, tile_count));
    } else {
        lb_store(my, lb_word(tag, kFlagAggregate, tile_count));
        int64_t look = tile - 1;
        uint32_t spins = 0;
        while (true) {
            const uint64_t w = lb_load(status + look * kRadixBins + d);
            const uint32_t wtag = (uint32_t)(w >> 34);
            const uint64_t flag = (w >> 32) & 3ull;
            if (wtag != (tag & 0x3FFFFFFFu) || flag == 0ull) {
                // every earlier tile is resident (it holds a smaller ticket) and
                // publishes without waiting; the bound only guards against a
                // broken invariant, turning it into a reported error
                if (++spins > (1u << 22)) {
                    raise_error(ctl, kBadInternal);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            excl += (uint32_t)w;
            if (flag == kFlagPrefix) break;
            --look;
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
// Run marking on the sorted keys.  Position j (occurrence o = vals[j]):
//   info[o] = -1 if its key occurs once, else j (its slot in the duplicate
//   buffer).  Runs of a repeated key are cut into pieces at multiples of
//   kChunk; each piece becomes a work item {start, len, key, kind}:
//     kind 0: the whole run -> sum and update the row directly;
//     kind 1: the run's first piece, the run continues past the window ->
//             partial sum to partB[window];
//     kind 2: a later piece, starting at a window boundary -> partA[window].
//   Every run with a kind-1 piece is also listed in longseg {head, key}.
// Distinct keys are counted per table, and occurrences in repeated rows.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_mark(Control* ctl, const uint32_t* __restrict__ keys,
                                                 const uint32_t* __restrict__ vals, int64_t m,
                                                 int64_t N, int32_t* __restrict__ info,
                                                 uint4* __restrict__ work,
                                                 uint2* __restrict__ longseg) {
    __shared__ uint32_t s_cnt[3];
    if (ctl->step_bad) return;
    if (threadIdx.x < 3) s_cnt[threadIdx.x] = 0u;
    __syncthreads();
    const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int lane = threadIdx.x & 63;
    bool emit = false, emit_long = false;
    uint4 rec = make_uint4(0, 0, 0, 0);
    if (j < m) {
        const uint32_t key = keys[j];
        const bool prev_same = j > 0 && keys[j - 1] == key;
        const bool next_same = j + 1 < m && keys[j + 1] == key;
        const bool dup = prev_same || next_same;
        const uint32_t o = vals[j];
        if ((int64_t)o < m) info[o] = dup ? (int32_t)j : -1;
        if (!prev_same) atomicAdd(&s_cnt[(int64_t)key >= N ? 0 : 1], 1u);
        if (dup) atomicAdd(&s_cnt[2], 1u);
        if (dup && (!prev_same || (j % kChunk) == 0)) {
            const int64_t win_end = (j / kChunk + 1) * kChunk;
            const int64_t lim = win_end < m ? win_end : m;
            int64_t e = j + 1;
            while (e < lim && keys[e] == key) ++e;
            const bool cont_after = (e == win_end) && (e < m) && keys[e] == key;
            uint32_t kind;
            if (!prev_same) kind = cont_after ? 1u : 0u;
            else kind = 2u;
            rec = make_uint4((uint32_t)j, (uint32_t)(e - j), key, kind);
            emit = true;
            emit_long = kind == 1u;
        }
    }
    // one atomic per wave for the work list
    const uint64_t em = __ballot(emit);
    if (em) {
        const int first = __ffsll((long long)em) - 1;
        uint32_t base = 0;
        if (lane == first) base = atomicAdd(&ctl->n_work, (uint32_t)__popcll(em));
        base = __shfl(base, first, 64);
        const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
        if (emit) work[base + __popcll(em & lt)] = rec;
    }
    if (emit_long) {
        const uint32_t slot = atomicAdd(&ctl->n_long, 1u);
        longseg[slot] = make_uint2(rec.x, rec.z);
    }
    __syncthreads();
    if (threadIdx.x < 3 && s_cnt[threadIdx.x]) {
        uint32_t* dstc = threadIdx.x == 0 ? &ctl->uniq_S : threadIdx.x == 1 ? &ctl->uniq_T
                                                                            : &ctl->dup_occ;
        atomicAdd(dstc, s_cnt[threadIdx.x]);
    }
}

hipError_t launch_mark(Control* ctl, const uint32_t* keys, const uint32_t* vals, int64_t m,
                       int64_t N, int32_t* info, uint4* work, uint2* longseg, hipStream_t s) {
    const int64_t blocks = (m + kBlock - 1) / kBlock;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_mark, dim3((unsigned)blocks), dim3(kBlock), 0, s, ctl, keys, vals, m, N,
                       info, work, longseg);
    return hipGetLastError();
}

}  // namespace huge
