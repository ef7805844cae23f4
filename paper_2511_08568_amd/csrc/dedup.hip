// Per-batch dedup + sort of row ids (a counting sort over the row-id domain).
//
// Each table owns a presence bitmap of ceil(N_t / 32) words in HBM.  A batch
// of ids is deduplicated by setting one bit per id; the distinct ids then come
// out in ascending order by scanning the bitmap: a block-wide popcount gives
// each 1024-word block its count, a per-table scan turns counts into offsets,
// and the emit pass writes every set bit's row at its rank.  For a forward the
// emit also stores, per non-zero word, (rank of its first set bit, the word,
// the forward's stamp), so the rank of any id of the batch is one load plus a
// popcount, and "was row r in the last batch" is one load.  Cost is
// O(ids + N_t / 32) with no comparison passes, which suits ids drawn from a
// bounded domain; the emit clears the bitmap behind it.
//
// Set-associative tables mark row r at bm_pos(r) = (set << qbits) | (r / nsets)
// instead of r, so U and PU come out grouped by set and ascending within each
// set (the order in which a set takes its events); the resident dump keeps
// plain row positions.
//
// Marking.  A table whose bitmap spans at most kOwnMaxSlices slices of
// kOwnSliceWords words is marked in LDS: one block per slice reads all of the
// table's ids, sets the bits that fall in its slice with LDS atomics, then
// stores the slice's non-zero words and the popcount of each of its bitmap
// blocks (so the count pass is not needed).  Its ids cost one 4-byte read per
// slice and the bitmap one write.  Larger tables are marked in HBM: Zipf-popular
// rows make many threads set the same bit, so each block first deduplicates its
// ids in a small LDS hash set and a popular row costs one device atomic per
// block instead of one per occurrence.  A bitmap word there is shared by blocks
// on every XCD, so that atomic (and the load before it) is served past the
// XCD's L2, a cache line per distinct id and block.
#include "launch.h"

namespace recmg {

constexpr int kLdsSet = 2048;  // entries of the per-block LDS set (power of two)
constexpr int kLdsProbes = 8;

__global__ void __launch_bounds__(kBlock) k_mark(DGlobal g, const int32_t *__restrict__ keys,
                                                 const int64_t *__restrict__ starts, int64_t n) {
    // The error word is read once per block: another block of this kernel may
    // set it meanwhile, and the waves of a block must agree before its barriers.
    __shared__ int s_err;
    if (threadIdx.x == 0) s_err = *g.err;
    __shared__ int64_t s_start[RECMG_MAX_TABLES + 1];
    __shared__ int64_t s_rows[RECMG_MAX_TABLES];
    __shared__ uint32_t *s_bm[RECMG_MAX_TABLES];
    __shared__ int32_t s_ns[RECMG_MAX_TABLES], s_qb[RECMG_MAX_TABLES];
    __shared__ bool s_own[RECMG_MAX_TABLES];
    __shared__ unsigned long long s_set[kLdsSet];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_start[t] = starts[t];
        if (t < g.T) {
            s_rows[t] = g.tabs[t].rows;
            s_bm[t] = g.tabs[t].bitmap;
            s_ns[t] = g.tabs[t].nsets;
            s_qb[t] = g.tabs[t].qbits;
            s_own[t] = owns_bitmap(g.tabs[t].bm_nblk);
        }
    }
    for (int k = threadIdx.x; k < kLdsSet; k += blockDim.x) s_set[k] = ~0ull;
    __syncthreads();
    if (s_err) return;  // block-uniform
    // each block takes a contiguous chunk, so repeats within the chunk meet in LDS
    const int64_t chunk = (n + gridDim.x - 1) / gridDim.x;
    const int64_t lo = (int64_t)blockIdx.x * chunk;
    const int64_t hi = lo + chunk < n ? lo + chunk : n;
    for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x) {
        const int t = find_seg(s_start, g.T, i);
        if (s_own[t]) continue;  // marked by k_mark_own
        const int32_t r = keys[i];
        if (r < 0 || (int64_t)r >= s_rows[t]) {
            atomicOr(g.err, ERR_RANGE);
            continue;
        }
        const unsigned long long key = ((unsigned long long)t << 32) | (uint32_t)r;
        bool mine = true;  // this thread must set the global bit
        uint32_t h = hash_row(r ^ (t * 0x9e3779b9)) & (kLdsSet - 1);
        for (int p = 0; p < kLdsProbes; ++p) {
            unsigned long long cur = s_set[h];
            if (cur == ~0ull) cur = atomicCAS(&s_set[h], ~0ull, key);
            if (cur == ~0ull) break;           // inserted here: mark globally
            if (cur == key) {                  // another thread of the block marks it
                mine = false;
                break;
            }
            h = (h + 1) & (kLdsSet - 1);
        }
        if (mine) {
            const uint32_t pos = bm_pos(s_ns[t], s_qb[t], r);
            uint32_t *w = s_bm[t] + (pos >> 5);
            const uint32_t bit = 1u << (pos & 31);
            if (!(__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & bit)) atomicOr(w, bit);
        }
    }
}

constexpr int kOwnThreads = 1024, kOwnUnroll = 8;
static_assert(kOwnSliceWords * 32 == 1 << 20, "a slice holds 2^20 bitmap positions");
static_assert(kOwnSliceBlocks <= kOwnThreads && kOwnSliceWords % kWordsPerBlock == 0, "slice = whole bitmap blocks");

// Block (slice, table) of the LDS marking: grid (g.own_slices, T); blocks of
// tables that are not owned, and slices past a table's bitmap, exit at once.
// Writes the slice's non-zero words into the (all-zero) bitmap and blocksum of
// each of its bitmap blocks.  Range errors are raised by slice 0 only.
__global__ void __launch_bounds__(kOwnThreads) k_mark_own(DGlobal g, const int32_t *__restrict__ keys,
                                                          const int64_t *__restrict__ starts) {
    __shared__ uint4 s_bm[kOwnSliceWords / 4];
    __shared__ int s_cnt[kOwnSliceBlocks];
    __shared__ int s_err;
    const int t = blockIdx.y, sl = blockIdx.x;
    const DTable &tb = g.tabs[t];
    const int nblk = tb.bm_nblk;
    if (!owns_bitmap(nblk) || sl * kOwnSliceBlocks >= nblk) return;  // block-uniform
    // the error word is read once: slice 0 of another table may set it meanwhile,
    // and the waves of the block must agree before its barriers
    if (threadIdx.x == 0) s_err = *g.err;
    const int sblk = nblk - sl * kOwnSliceBlocks < kOwnSliceBlocks ? nblk - sl * kOwnSliceBlocks : kOwnSliceBlocks;
    const int nq = sblk * (kWordsPerBlock / 4);  // uint4 words of the slice
    for (int k = threadIdx.x; k < nq; k += kOwnThreads) s_bm[k] = make_uint4(0u, 0u, 0u, 0u);
    if (threadIdx.x < kOwnSliceBlocks) s_cnt[threadIdx.x] = 0;
    __syncthreads();
    if (s_err) return;  // block-uniform
    uint32_t *bm = reinterpret_cast<uint32_t *>(s_bm);
    const int64_t lo = starts[t], hi = starts[t + 1];
    const int64_t rows = tb.rows;
    const int32_t ns = tb.nsets, qb = tb.qbits;
    for (int64_t i0 = lo + threadIdx.x; i0 < hi; i0 += (int64_t)kOwnThreads * kOwnUnroll) {
        int32_t r[kOwnUnroll];
#pragma unroll
        for (int u = 0; u < kOwnUnroll; ++u) {
            const int64_t i = i0 + (int64_t)u * kOwnThreads;
            r[u] = i < hi ? keys[i] : 0;
        }
#pragma unroll
        for (int u = 0; u < kOwnUnroll; ++u) {
            if (i0 + (int64_t)u * kOwnThreads >= hi) continue;
            if (r[u] < 0 || (int64_t)r[u] >= rows) {
                if (sl == 0) atomicOr(g.err, ERR_RANGE);
                continue;
            }
            const uint32_t pos = bm_pos(ns, qb, r[u]);
            if ((int)(pos >> 20) != sl) continue;  // the position's slice
            const uint32_t w = (pos >> 5) & (kOwnSliceWords - 1), bit = 1u << (pos & 31);
            if (!(bm[w] & bit)) atomicOr(&bm[w], bit);
        }
    }
    __syncthreads();
    uint4 *gbm = reinterpret_cast<uint4 *>(tb.bitmap + (int64_t)sl * kOwnSliceWords);
    for (int k = threadIdx.x; k < nq; k += kOwnThreads) {
        const uint4 v = s_bm[k];
        if (v.x | v.y | v.z | v.w) gbm[k] = v;
        int c = __popc(v.x) + __popc(v.y) + __popc(v.z) + __popc(v.w);
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) c += __shfl_xor(c, m);
        // a wave's 64 uint4 words lie in one bitmap block of 256 uint4 words
        if ((threadIdx.x & 63) == 0 && c) atomicAdd(&s_cnt[k / (kWordsPerBlock / 4)], c);
    }
    __syncthreads();
    if (threadIdx.x < sblk) g.blocksum[tb.bm_block0 + sl * kOwnSliceBlocks + threadIdx.x] = s_cnt[threadIdx.x];
}

// Mark the resident rows of every table (for the sorted dump).
__global__ void __launch_bounds__(kBlock) k_mark_resident(DGlobal g) {
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < tb.cap;
         k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t r = tb.slot_row[k];
        if (r >= 0) atomicOr(tb.bitmap + (r >> 5), 1u << (r & 31));
    }
}

__device__ __forceinline__ int block_table(const DGlobal &g, int blk) {
    __shared__ int s_t;
    if (threadIdx.x == 0) s_t = find_seg32(g.bm_block_start, g.T, blk);
    __syncthreads();
    return s_t;
}

__global__ void __launch_bounds__(kBlock) k_bm_count(DGlobal g) {
    if (*g.err) return;
    __shared__ int tmp[16];
    const int blk = blockIdx.x;
    const int t = block_table(g, blk);
    const DTable &tb = g.tabs[t];
    const int64_t w0 = (int64_t)(blk - tb.bm_block0) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
    const uint4 w = *reinterpret_cast<const uint4 *>(tb.bitmap + w0);
    const int c = __popc(w.x) + __popc(w.y) + __popc(w.z) + __popc(w.w);
    const int s = block_sum(c, tmp);
    if (threadIdx.x == 0) g.blocksum[blk] = s;
}

// One block per table: exclusive scan of the table's block counts.
// counts[t * count_stride] receives the table's total.
__global__ void __launch_bounds__(1024) k_bm_scan(DGlobal g, int32_t *counts, int count_stride) {
    if (*g.err) return;
    __shared__ int tmp[16];
    const int t = blockIdx.x;
    const int b0 = g.bm_block_start[t], nb = g.bm_block_start[t + 1] - b0;
    int carry = 0;
    for (int base = 0; base < nb; base += blockDim.x) {
        const int k = base + threadIdx.x;
        const int v = k < nb ? g.blocksum[b0 + k] : 0;
        int tot;
        const int ex = block_excl_scan(v, tmp, &tot);
        if (k < nb) g.blockoff[b0 + k] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) counts[(int64_t)t * count_stride] = carry;
}

// Write the distinct ids in ascending order (U, PU or the resident dump).
template <int MODE>
__global__ void __launch_bounds__(kBlock) k_bm_emit(DGlobal g, int32_t stamp) {
    if (*g.err) return;
    __shared__ int tmp[16];
    const int blk = blockIdx.x;
    const int t = block_table(g, blk);
    const DTable &tb = g.tabs[t];
    const int64_t wbase = (int64_t)(blk - tb.bm_block0) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
    const uint4 w4 = *reinterpret_cast<const uint4 *>(tb.bitmap + wbase);
    const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
    const int cnt = __popc(w[0]) + __popc(w[1]) + __popc(w[2]) + __popc(w[3]);
    int tot;
    const int first = g.blockoff[blk] + block_excl_scan(cnt, tmp, &tot);
    if (tot == 0) return;  // block-uniform
    int32_t *out;
    if (MODE == EMIT_FORWARD) out = g.U + g.tstart[t];
    else if (MODE == EMIT_PREFETCH) out = g.PU + g.pstart[t];
    else out = g.dump + tb.cap_off;
    int u = first;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t bits = w[q];
        if (!bits) continue;
        const int64_t word = wbase + q;
        if (MODE == EMIT_FORWARD) tb.rank[word] = make_uint4((uint32_t)u, bits, (uint32_t)stamp, 0u);
        tb.bitmap[word] = 0;
        while (bits) {
            const int b = __ffs(bits) - 1;
            bits &= bits - 1;
            const uint32_t pos = (uint32_t)(word * 32 + b);
            out[u++] = MODE == EMIT_DUMP ? (int32_t)pos : bm_row(tb, pos);
        }
    }
}

// Small tables: count, scan and emit in one kernel, one block of 1024 threads
// per table walking its bitmap 4096 words at a time (the three-kernel form
// costs two more launches, which dominate when a table's bitmap is a few
// blocks: configuration 1 has four).
constexpr int kFusedThreads = 1024, kFusedWords = kFusedThreads * kWordsPerThread;

template <int MODE>
__global__ void __launch_bounds__(kFusedThreads) k_bm_fused(DGlobal g, int32_t *counts, int count_stride,
                                                           int32_t stamp) {
    if (*g.err) return;
    __shared__ int tmp[16];
    const int t = blockIdx.x;
    const DTable &tb = g.tabs[t];
    int32_t *out;
    if (MODE == EMIT_FORWARD) out = g.U + g.tstart[t];
    else if (MODE == EMIT_PREFETCH) out = g.PU + g.pstart[t];
    else out = g.dump + tb.cap_off;
    int base = 0;  // distinct ids of the words before this pass
    for (int64_t w0 = 0; w0 < tb.bm_words; w0 += kFusedWords) {
        const int64_t wbase = w0 + threadIdx.x * kWordsPerThread;
        uint32_t w[4] = {0u, 0u, 0u, 0u};
        if (wbase < tb.bm_words) {  // bm_words is a multiple of kWordsPerBlock, so four words are present
            const uint4 w4 = *reinterpret_cast<const uint4 *>(tb.bitmap + wbase);
            w[0] = w4.x, w[1] = w4.y, w[2] = w4.z, w[3] = w4.w;
        }
        const int cnt = __popc(w[0]) + __popc(w[1]) + __popc(w[2]) + __popc(w[3]);
        int tot;
        int u = base + block_excl_scan(cnt, tmp, &tot);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t bits = w[q];
            if (!bits) continue;
            const int64_t word = wbase + q;
            if (MODE == EMIT_FORWARD) tb.rank[word] = make_uint4((uint32_t)u, bits, (uint32_t)stamp, 0u);
            tb.bitmap[word] = 0;
            while (bits) {
                const int b = __ffs(bits) - 1;
                bits &= bits - 1;
                const uint32_t pos = (uint32_t)(word * 32 + b);
                out[u++] = MODE == EMIT_DUMP ? (int32_t)pos : bm_row(tb, pos);
            }
        }
        base += tot;
    }
    if (threadIdx.x == 0) counts[(int64_t)t * count_stride] = base;
}

// ------------------------------------------------------------------- launchers

static inline unsigned grid_for(int64_t n, int per_block, unsigned cap) {
    int64_t b = (n + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > (int64_t)cap) b = cap;
    return (unsigned)b;
}

void launch_mark(const DGlobal &g, const int32_t *keys, const int64_t *starts, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    if (g.own_tables > 0) k_mark_own<<<dim3((unsigned)g.own_slices, (unsigned)g.T), kOwnThreads, 0, s>>>(g, keys, starts);
    if (g.own_tables < g.T) k_mark<<<grid_for(n, kBlock * 8, 4096), kBlock, 0, s>>>(g, keys, starts, n);
}

void launch_mark_resident(const DGlobal &g, int32_t max_cap, hipStream_t s) {
    if (max_cap <= 0) return;
    dim3 grid(grid_for(max_cap, kBlock * 4, 4096), g.T);
    k_mark_resident<<<grid, kBlock, 0, s>>>(g);
}

void launch_dedup(const DGlobal &g, int mode, int32_t *counts, int count_stride, int32_t stamp, int32_t max_nblk,
                  hipStream_t s) {
    if (max_nblk <= kFusedMaxBlocks) {
        if (mode == EMIT_FORWARD) k_bm_fused<EMIT_FORWARD><<<g.T, kFusedThreads, 0, s>>>(g, counts, count_stride, stamp);
        else if (mode == EMIT_PREFETCH) k_bm_fused<EMIT_PREFETCH><<<g.T, kFusedThreads, 0, s>>>(g, counts, count_stride, stamp);
        else k_bm_fused<EMIT_DUMP><<<g.T, kFusedThreads, 0, s>>>(g, counts, count_stride, stamp);
        return;
    }
    // k_mark_own has counted the owned tables' blocks (not those of the resident dump)
    if (mode == EMIT_DUMP || g.own_tables < g.T) k_bm_count<<<g.total_bm_blocks, kBlock, 0, s>>>(g);
    k_bm_scan<<<g.T, 1024, 0, s>>>(g, counts, count_stride);
    if (mode == EMIT_FORWARD) k_bm_emit<EMIT_FORWARD><<<g.total_bm_blocks, kBlock, 0, s>>>(g, stamp);
    else if (mode == EMIT_PREFETCH) k_bm_emit<EMIT_PREFETCH><<<g.total_bm_blocks, kBlock, 0, s>>>(g, stamp);
    else k_bm_emit<EMIT_DUMP><<<g.total_bm_blocks, kBlock, 0, s>>>(g, stamp);
}

}  // namespace recmg
