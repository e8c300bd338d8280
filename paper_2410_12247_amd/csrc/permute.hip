// Dispatch: histogram, scan, stable scatter and row gather.
//
// Order of rows: (bucket ascending, slot ascending).  A bucket is the local
// expert, or, when the pipeline cuts token ranges, token-range stage * EL +
// local expert.  A token selects an expert at most once, so slot order
// within an expert is token order (the order of the paper's Fig. 7a
// example).  Three passes, no atomics (one kernel doing all three in one
// wave when the slots fit one chunk):
//   1. one wave per chunk of kPermChunk slots: wave-level match (nine
//      ballots on the bucket id) gives each slot its rank among the equal
//      ids before it in the 64-slot step, a per-chunk LDS counter carries the
//      rank across steps -> slot_rank, and chunk_counts[chunk][b];
//   2. one workgroup: per-bucket exclusive scan over chunks -> chunk_base,
//      counts, and a wave-level (DPP row shifts + readlane) scan over
//      buckets -> offsets (and the rows per local expert over stages);
//   3. one thread per slot: row = offsets[b] + chunk_base[chunk][b] +
//      slot_rank -> sorted_slot[row], slot_row[slot].
// The gather copies whole rows with 16-byte loads and stores, one wave per
// row.
#include "common.h"

namespace moe {
namespace {

// Bucket of slot s (token s / k) for local expert e, or -1 when not local.
__device__ __forceinline__ int slot_bucket(const int32_t *ids, int64_t s, int k, int e0, int EL,
                                           int64_t tps) {
    int e = ids[s] - e0;
    if (e < 0 || e >= EL) return -1;
    if (tps > 0) e += (int)((s / k) / tps) * EL;
    return e;
}

__global__ __launch_bounds__(64) void hist_kernel(const int32_t *__restrict__ ids, int64_t nslots,
                                                  int k, int e0, int EL, int64_t tps, int NB,
                                                  int32_t *__restrict__ chunk_counts,
                                                  int32_t *__restrict__ slot_rank) {
    __shared__ int cnt[kMaxExperts];
    const int lane = threadIdx.x;
    for (int e = lane; e < NB; e += 64) cnt[e] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kPermChunk;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    // every id of the chunk is loaded before the first is ranked: one memory
    // round trip per chunk instead of one per 64 slots
    // (unconditional loads of a clamped slot, kept above the compiler
    // barrier so that they are not sunk back to their uses)
    constexpr int NIT = kPermChunk / 64;
    int idv[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) idv[it] = ids[min<int64_t>(base + it * 64 + lane, nslots - 1)];
    asm volatile("" ::: "memory");
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int64_t s = base + it * 64 + lane;
        int e = idv[it] - e0;
        if (s >= nslots || e < 0 || e >= EL) e = -1;
        else if (tps > 0) e += (int)((uint32_t)s / (uint32_t)k / (uint32_t)tps) * EL;  // s < 2^31
        // lanes holding the same value (e + 1 in [0, 256], nine bits)
        const uint32_t v = (uint32_t)(e + 1);
        uint64_t match = ~0ull;
#pragma unroll
        for (int b = 0; b < 9; ++b) {
            const bool bit = (v >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            match &= bit ? bal : ~bal;
        }
        const int before = __popcll(match & lt_mask);
        if (e >= 0) {
            slot_rank[s] = cnt[e] + before;
        }
        // the lowest lane of each group advances that expert's counter; all
        // reads above were issued first (one wave, LDS operations in order)
        __syncthreads();
        if (e >= 0 && before == 0) cnt[e] += __popcll(match);
        __syncthreads();
    }
    for (int e = lane; e < NB; e += 64) chunk_counts[(int64_t)blockIdx.x * NB + e] = cnt[e];
}

// Inclusive scan over a wave: DPP row_shr 1, 2, 4, 8 inside each 16-lane row
// (lanes with no source add 0), then row totals carried with readlane.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
    const int lane = threadIdx.x & 63;
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
    const int r0 = __builtin_amdgcn_readlane(v, 15);
    const int r1 = __builtin_amdgcn_readlane(v, 31);
    const int r2 = __builtin_amdgcn_readlane(v, 47);
    const int row = lane >> 4;
    v += (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
    return v;
}

__global__ __launch_bounds__(256) void scan_kernel(const int32_t *__restrict__ chunk_counts,
                                                   int64_t nchunks, int NB, int EL,
                                                   int32_t *__restrict__ chunk_base,
                                                   int32_t *__restrict__ counts,
                                                   int32_t *__restrict__ offsets,
                                                   int32_t *__restrict__ counts_el) {
    __shared__ int wave_tot[4];
    __shared__ int totals[kMaxExperts];
    const int e = threadIdx.x;
    int run = 0;
    if (e < NB) {
        // sixteen chunks' counts loaded before they are summed, so a long
        // chunk list costs nchunks / 16 memory round trips, not nchunks
        constexpr int U = 16;
        int64_t c = 0;
        for (; c + U <= nchunks; c += U) {
            int v[U];
#pragma unroll
            for (int i = 0; i < U; ++i) v[i] = chunk_counts[(c + i) * NB + e];
#pragma unroll
            for (int i = 0; i < U; ++i) {
                chunk_base[(c + i) * NB + e] = run;
                run += v[i];
            }
        }
        for (; c < nchunks; ++c) {
            const int v = chunk_counts[c * NB + e];
            chunk_base[c * NB + e] = run;
            run += v;
        }
        counts[e] = run;
        totals[e] = run;
    }
    const int incl = wave_inclusive_scan(e < NB ? run : 0);
    const int w = e >> 6;
    if ((e & 63) == 63) wave_tot[w] = incl;
    __syncthreads();
    int carry = 0;
    for (int i = 0; i < w; ++i) carry += wave_tot[i];
    if (e < NB) offsets[e] = carry + incl - run;
    if (e == NB - 1) offsets[NB] = carry + incl;
    if (counts_el && e < EL) {  // rows per local expert over the stages
        int sum = 0;
        for (int b = e; b < NB; b += EL) sum += totals[b];
        counts_el[e] = sum;
    }
}

__global__ __launch_bounds__(256) void scatter_kernel(const int32_t *__restrict__ ids,
                                                      int64_t nslots, int k, int e0, int EL,
                                                      int64_t tps, int NB,
                                                      const int32_t *__restrict__ chunk_base,
                                                      const int32_t *__restrict__ slot_rank,
                                                      const int32_t *__restrict__ offsets,
                                                      int32_t *__restrict__ sorted_slot,
                                                      int32_t *__restrict__ slot_row) {
    const int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (s >= nslots) return;
    const int e = slot_bucket(ids, s, k, e0, EL, tps);
    if (e < 0) {
        slot_row[s] = -1;
        return;
    }
    const int64_t chunk = s / kPermChunk;
    const int row = offsets[e] + chunk_base[chunk * NB + e] + slot_rank[s];
    sorted_slot[row] = (int32_t)s;
    slot_row[s] = row;
}

// The three passes in one wave for at most kPermChunk slots (one chunk:
// decode batches), one launch instead of three: the ranks as in
// hist_kernel, kept in registers; the bucket scan as in scan_kernel, 64
// buckets at a time with a carry; then the rows.  Same counts, offsets and
// rows as the three kernels.
__global__ __launch_bounds__(64) void dispatch_one_chunk_kernel(
    const int32_t *__restrict__ ids, int64_t nslots, int k, int e0, int EL, int64_t tps, int NB,
    int32_t *__restrict__ counts, int32_t *__restrict__ offsets,
    int32_t *__restrict__ counts_el, int32_t *__restrict__ sorted_slot,
    int32_t *__restrict__ slot_row) {
    __shared__ int cnt[kMaxExperts];
    __shared__ int off[kMaxExperts];
    const int lane = threadIdx.x;
    for (int e = lane; e < NB; e += 64) cnt[e] = 0;
    __syncthreads();
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    constexpr int NIT = kPermChunk / 64;
    // groups of 64 slots that hold any (the rest of the unrolled loops is
    // skipped: decode batches have one or two)
    const int nit = (int)((nslots + 63) / 64);
    int idv[NIT], bucket[NIT], rank[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) idv[it] = ids[min<int64_t>(it * 64 + lane, nslots - 1)];
    asm volatile("" ::: "memory");
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        bucket[it] = -1;
        rank[it] = 0;
        if (it >= nit) continue;
        const int s = it * 64 + lane;
        int e = idv[it] - e0;
        if (s >= nslots || e < 0 || e >= EL) e = -1;
        else if (tps > 0) e += (int)((uint32_t)s / (uint32_t)k / (uint32_t)tps) * EL;
        const uint32_t v = (uint32_t)(e + 1);
        uint64_t match = ~0ull;
#pragma unroll
        for (int b = 0; b < 9; ++b) {
            const bool bit = (v >> b) & 1u;
            const uint64_t bal = __ballot(bit);
            match &= bit ? bal : ~bal;
        }
        const int before = __popcll(match & lt_mask);
        bucket[it] = e;
        rank[it] = e >= 0 ? cnt[e] + before : 0;
        __syncthreads();
        if (e >= 0 && before == 0) cnt[e] += __popcll(match);
        __syncthreads();
    }
    int carry = 0;
    for (int b0 = 0; b0 < NB; b0 += 64) {
        const int e = b0 + lane;
        const int v = e < NB ? cnt[e] : 0;
        const int incl = wave_inclusive_scan(v);
        if (e < NB) {
            counts[e] = v;
            off[e] = carry + incl - v;
            offsets[e] = carry + incl - v;
        }
        carry += __builtin_amdgcn_readlane(incl, 63);
    }
    if (lane == 0) offsets[NB] = carry;
    if (counts_el) {  // rows per local expert over the stages
        for (int e = lane; e < EL; e += 64) {
            int sum = 0;
            for (int b = e; b < NB; b += EL) sum += cnt[b];
            counts_el[e] = sum;
        }
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int s = it * 64 + lane;
        if (it < nit && s < nslots) {
            const int e = bucket[it];
            if (e < 0) {
                slot_row[s] = -1;
            } else {
                const int row = off[e] + rank[it];
                sorted_slot[row] = s;
                slot_row[s] = row;
            }
        }
    }
}

// One wave per row; rows [offsets[e_first], offsets[e_first+e_count]).
__global__ __launch_bounds__(256) void gather_kernel(const int32_t *__restrict__ offsets,
                                                     int e_first, int e_count,
                                                     const int32_t *__restrict__ sorted_slot,
                                                     int k, int H, const bf16_t *__restrict__ x,
                                                     bf16_t *__restrict__ x_perm) {
    const int r_begin = offsets[e_first];
    const int r_end = offsets[e_first + e_count];
    const int lane = threadIdx.x & 63;
    const int wave = (int)(blockIdx.x * 4 + (threadIdx.x >> 6));
    const int nwaves = (int)(gridDim.x * 4);
    const int vecs = H / 8;  // 16-byte vectors per row
    for (int r = r_begin + wave; r < r_end; r += nwaves) {
        const int64_t t = sorted_slot[r] / k;
        const uint4 *src = reinterpret_cast<const uint4 *>(x + t * H);
        uint4 *dst = reinterpret_cast<uint4 *>(x_perm + (int64_t)r * H);
        for (int v = lane; v < vecs; v += 64) dst[v] = src[v];
    }
}

}  // namespace

hipError_t launch_permute(const moe_dims &d, const int32_t *ids, void *ws, const WsLayout &L,
                          int64_t tokens_per_stage, int32_t *counts, int32_t *offsets,
                          int32_t *counts_el, int32_t *sorted_slot, int32_t *slot_row,
                          hipStream_t s) {
    char *base = static_cast<char *>(ws);
    int32_t *chunk_counts = reinterpret_cast<int32_t *>(base + L.chunk_counts);
    int32_t *chunk_base = reinterpret_cast<int32_t *>(base + L.chunk_base);
    int32_t *slot_rank = reinterpret_cast<int32_t *>(base + L.slot_rank);
    const int64_t nslots = d.tokens * d.top_k;
    const int64_t tps = tokens_per_stage;
    const int NB = L.nbuckets;
    if (nslots <= kPermChunk) {
        dispatch_one_chunk_kernel<<<1, 64, 0, s>>>(ids, nslots, d.top_k, d.local_begin,
                                                    d.local_count, tps, NB, counts, offsets,
                                                    tps > 0 ? counts_el : nullptr, sorted_slot,
                                                    slot_row);
        return hipGetLastError();
    }
    hist_kernel<<<(unsigned)L.nchunks, 64, 0, s>>>(ids, nslots, d.top_k, d.local_begin,
                                                    d.local_count, tps, NB, chunk_counts,
                                                    slot_rank);
    scan_kernel<<<1, 256, 0, s>>>(chunk_counts, L.nchunks, NB, d.local_count, chunk_base, counts,
                                  offsets, tps > 0 ? counts_el : nullptr);
    scatter_kernel<<<(unsigned)((nslots + 255) / 256), 256, 0, s>>>(
        ids, nslots, d.top_k, d.local_begin, d.local_count, tps, NB, chunk_base, slot_rank,
        offsets, sorted_slot, slot_row);
    return hipGetLastError();
}

hipError_t launch_gather(const moe_dims &d, int e_first, int e_count, const int32_t *offsets,
                         const int32_t *sorted_slot, const bf16_t *x, bf16_t *x_perm,
                         int64_t max_rows, hipStream_t s) {
    if (e_count <= 0 || max_rows <= 0) return hipSuccess;
    int64_t blocks = (max_rows + 3) / 4;
    if (blocks > 4096) blocks = 4096;
    gather_kernel<<<(unsigned)blocks, 256, 0, s>>>(offsets, e_first, e_count, sorted_slot,
                                                   d.top_k, d.hidden, x, x_perm);
    return hipGetLastError();
}

}  // namespace moe
