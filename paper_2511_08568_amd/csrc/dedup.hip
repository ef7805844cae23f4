// Per-batch dedup + sort of row ids (a counting sort over the row-id domain).
//
// Each table owns a presence bitmap of ceil(N_t / 32) words in HBM.  A batch
// of ids is deduplicated by setting one bit per id; the distinct ids then come
// out in ascending order by scanning the bitmap: a block-wide popcount gives
// each 1024-word block its count, a per-table scan turns counts into offsets,
// and the emit pass writes every set bit's row at its rank.  For every
// non-zero word the emit also stores (rank of its first bit, the word), so the
// rank of any id in the distinct list is one load plus a popcount.  Cost is
// O(ids + N_t / 32) with no comparison passes, which suits ids drawn from a
// bounded domain; the emit clears the bitmap behind it.
//
// The emit runs one of three visitors on every distinct id:
//   EMIT_FORWARD  probe the row -> slot map (the lookup's cache probe), count
//                 hits, stamp hit slots, number the misses;
//   EMIT_PREFETCH classify a prefetch id as resident / missed by the last
//                 batch / new candidate (Alg. 1's prefetch loop, as a set);
//   EMIT_DUMP     write the sorted resident rows for recmg_stats.
#include "launch.h"

namespace recmg {

// ------------------------------------------------------------------- mark

__global__ void __launch_bounds__(kBlock) k_mark(DGlobal g, const int32_t *__restrict__ keys,
                                                 const int64_t *__restrict__ starts, int64_t n) {
    if (*g.err) return;
    __shared__ int64_t s_start[RECMG_MAX_TABLES + 1];
    __shared__ int64_t s_rows[RECMG_MAX_TABLES];
    __shared__ uint32_t *s_bm[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_start[t] = starts[t];
        if (t < g.T) {
            s_rows[t] = g.tabs[t].rows;
            s_bm[t] = g.tabs[t].bitmap;
        }
    }
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        const int t = find_seg(s_start, g.T, i);
        const int32_t r = keys[i];
        if (r < 0 || (int64_t)r >= s_rows[t]) {
            atomicOr(g.err, ERR_RANGE);
            continue;
        }
        uint32_t *w = s_bm[t] + (r >> 5);
        const uint32_t bit = 1u << (r & 31);
        if (!(__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & bit)) atomicOr(w, bit);
    }
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

// ------------------------------------------------------------------- count

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

// ------------------------------------------------------------------- emit

enum { EMIT_FORWARD = 0, EMIT_PREFETCH = 1, EMIT_DUMP = 2 };

struct EmitCtx {
    int32_t stamp;     // EMIT_FORWARD: stamp of this forward
    int32_t have_fwd;  // EMIT_PREFETCH: a forward ran since the last placement
};

template <int MODE>
__global__ void __launch_bounds__(kBlock) k_bm_emit(DGlobal g, EmitCtx ctx) {
    if (*g.err) return;
    __shared__ int tmp[16];
    __shared__ int s_base;
    const int blk = blockIdx.x;
    const int t = block_table(g, blk);
    const DTable &tb = g.tabs[t];
    TState &st = g.st[t];
    const int64_t wbase = (int64_t)(blk - tb.bm_block0) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
    uint4 w4 = *reinterpret_cast<const uint4 *>(tb.bitmap + wbase);
    uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
    const int cnt = __popc(w[0]) + __popc(w[1]) + __popc(w[2]) + __popc(w[3]);
    int tot;
    const int first = g.blockoff[blk] + block_excl_scan(cnt, tmp, &tot);
    if (tot == 0) return;  // block-uniform

    int64_t seg;  // where table t's distinct ids start in the output arrays
    if (MODE == EMIT_FORWARD) seg = g.tstart[t];
    else if (MODE == EMIT_PREFETCH) seg = g.pstart[t];
    else seg = tb.cap_off;

    int hits = 0, hits_pf = 0, pres = 0, nappend = 0;
    // pass 1: rank words, emit rows, run the visitor
    int u = first;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        uint32_t bits = w[q];
        if (!bits) continue;
        const int64_t word = wbase + q;
        if (MODE == EMIT_FORWARD) tb.rank[word] = make_uint2((uint32_t)u, bits);
        tb.bitmap[word] = 0;
        while (bits) {
            const int b = __ffs(bits) - 1;
            bits &= bits - 1;
            const int32_t row = (int32_t)(word * 32 + b);
            if (MODE == EMIT_FORWARD) {
                g.U[seg + u] = row;
                const int32_t slot = map_find(tb, row);
                if (slot >= 0) {
                    g.slotU[seg + u] = slot;
                    tb.slot_touch[slot] = ctx.stamp;
                    ++hits;
                    hits_pf += (tb.slot_flags[slot] & F_PF) ? 1 : 0;
                } else {
                    g.slotU[seg + u] = kPending;
                    ++nappend;
                }
            } else if (MODE == EMIT_PREFETCH) {
                int32_t tag = -1;  // the row itself if it becomes a new candidate
                const int32_t slot = map_find(tb, row);
                if (slot >= 0) {
                    atomicOr(&tb.slot_flags[slot], F_INP);
                    ++pres;
                } else {
                    int64_t m = -1;
                    if (ctx.have_fwd) {
                        // was it missed by the last batch?  U of that batch is sorted.
                        const int64_t ts = g.tstart[t];
                        int lo = 0, hi = st.ucount;
                        while (lo < hi) {
                            const int mid = (lo + hi) >> 1;
                            if (g.U[ts + mid] < row) lo = mid + 1;
                            else hi = mid;
                        }
                        if (lo < st.ucount && g.U[ts + lo] == row) m = -(int64_t)g.slotU[ts + lo] - 1;
                        if (m >= 0) atomicOr(&g.mflags[ts + m], F_INP);
                    }
                    if (m < 0) {
                        tag = row;
                        ++nappend;
                    }
                }
                g.ptag[seg + u] = tag;
            } else {
                g.dump[seg + u] = row;
            }
            ++u;
        }
    }
    if (MODE == EMIT_DUMP) return;

    // pass 2: number the appended ids (misses / new candidates) block-wide
    const int app_ex = block_excl_scan(nappend, tmp, &tot);
    if (threadIdx.x == 0 && tot > 0)
        s_base = atomicAdd(MODE == EMIT_FORWARD ? &st.mcount : &st.npcount, tot);
    __syncthreads();
    if (nappend) {
        int a = s_base + app_ex;
        for (int k = first; k < first + cnt; ++k) {
            if (MODE == EMIT_FORWARD) {
                if (g.slotU[seg + k] == kPending) {
                    g.slotU[seg + k] = -(a + 1);
                    g.M[seg + a] = g.U[seg + k];
                    g.mflags[seg + a] = 0;
                    ++a;
                }
            } else {
                const int32_t row = g.ptag[seg + k];
                if (row >= 0) g.NP[seg + a++] = row;
            }
        }
    }
    if (MODE == EMIT_FORWARD) {
        const int h = block_sum(hits, tmp);
        const int hp = block_sum(hits_pf, tmp);
        if (threadIdx.x == 0) {
            if (h) atomicAdd(&st.hits, h);
            if (hp) atomicAdd(&st.hits_pf, hp);
        }
    } else {
        const int p = block_sum(pres, tmp);
        if (threadIdx.x == 0 && p) atomicAdd(&st.p_res, p);
    }
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
    k_mark<<<grid_for(n, kBlock * 4, 16384), kBlock, 0, s>>>(g, keys, starts, n);
}

void launch_mark_resident(const DGlobal &g, int32_t max_cap, hipStream_t s) {
    if (max_cap <= 0) return;
    dim3 grid(grid_for(max_cap, kBlock * 4, 4096), g.T);
    k_mark_resident<<<grid, kBlock, 0, s>>>(g);
}

void launch_dedup(const DGlobal &g, int mode, int32_t *counts, int count_stride, int32_t stamp, int32_t have_fwd,
                  hipStream_t s) {
    k_bm_count<<<g.total_bm_blocks, kBlock, 0, s>>>(g);
    k_bm_scan<<<g.T, 1024, 0, s>>>(g, counts, count_stride);
    EmitCtx ctx{stamp, have_fwd};
    if (mode == EMIT_FORWARD) k_bm_emit<EMIT_FORWARD><<<g.total_bm_blocks, kBlock, 0, s>>>(g, ctx);
    else if (mode == EMIT_PREFETCH) k_bm_emit<EMIT_PREFETCH><<<g.total_bm_blocks, kBlock, 0, s>>>(g, ctx);
    else k_bm_emit<EMIT_DUMP><<<g.total_bm_blocks, kBlock, 0, s>>>(g, ctx);
}

}  // namespace recmg
