// Placement between batches: the batched form of Alg. 1 (load_embeddings)
// and Alg. 2 (gpu_buffer_populate), Sec. VI-B.
//
// Per table t the candidate set is K = R ∪ M ∪ set(P): resident slots, the
// last batch's misses (already in HBM staging) and the prefetch list.  Every
// member gets a score (aging, touch, prefetch, below), and the cache keeps the
// min(Cap, |K|) largest keys (score, row).  Instead of one victim scan per
// insertion, one radix select per placement finds the threshold key: 11-bit
// digits from the top, each pass a histogram kernel and a one-block-per-table
// kernel that picks the digit holding the Cap-th largest key.  Keys are
// distinct (rows are distinct), so exactly min(Cap, |K|) keys are >= the
// threshold.
//
// Scores:  LRU_BATCH  touched by the last batch: lru_touch; prefetched:
//                     max(score, pscore) with pscore = lru_touch + 1
//          LFU_BATCH  every row's score is its batch count (k_plc_freq adds
//                     the last batch); a prefetch does not change it
//          PRIORITY   residents first age by one, saturating at 0 (Alg. 2);
//                     touched: caching bit + ES (Alg. 1); prefetched:
//                     max(score, ES); a touched resident loses its prefetch flag.
//
// Kernels on the stream: k_plc_prep, [k_plc_bits], dedup of P with the
// EMIT_PREFETCH visitor (dedup.hip), k_plc_update (scores + histogram of
// pass 0), k_plc_pick, { k_plc_select (histogram of pass 1..), k_plc_pick }*,
// k_plc_evict, k_map_clear / k_map_refill (rebuild
// when deleted entries pile up), k_plc_admit, k_plc_fill, k_plc_finalize.
#include <hip/hip_ext.h>

#include "launch.h"

namespace recmg {

__global__ void k_plc_prep(DGlobal g, const int64_t *__restrict__ poff, int64_t np, int32_t have_fwd) {
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        const int64_t v = poff[t];
        g.pstart[t] = v;
        // table t's fill list lives at ftstart[t] + pstart[t] and holds at most
        // (its last-batch indices) + (its prefetch ids) entries
        g.ftstart[t] = have_fwd ? g.tstart[t] : 0;
        if (t < g.T && v > poff[t + 1]) atomicOr(g.err, ERR_OFFSETS);
        if ((t == 0 && v != 0) || (t == g.T && v != np)) atomicOr(g.err, ERR_OFFSETS);
        if (t < g.T) {
            TState &st = g.st[t];
            st.pcount = 0;
            st.npcount = 0;
            st.popped = 0;
            st.p_res = 0;
            st.evicted = 0;
            st.adm_miss = 0;
            st.p_fill = 0;
            st.p_drop = 0;
            st.m_drop = 0;
            st.z1_keys = 0;
            st.pend_keep = 0;
            // set-associative tables and resident rings update the digest by
            // the rows that come and go
            st.digest_acc = (g.tabs[t].ways || g.tabs[t].ring_cap) ? st.digest : 0ull;
        }
    }
}

// Caching bits of the last batch, OR-ed per row into a byte of the slot (hit)
// or of the miss entry.  Every writer stores the same value 1, so plain byte
// stores suffice (no read-modify-write atomics on popular rows).
__global__ void __launch_bounds__(kBlock) k_plc_bits(DGlobal g, const uint8_t *__restrict__ bits, int64_t n) {
    if (*g.err) return;
    __shared__ int64_t s_start[RECMG_MAX_TABLES + 1];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) s_start[t] = g.tstart[t];
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        if (!bits[i]) continue;
        const int t = find_seg(s_start, g.T, i);
        const int32_t s = g.src[i];
        uint8_t *f = s >= 0 ? &g.tabs[t].slot_cbit[s] : &g.mcbit[s_start[t] + (-(int64_t)s - 1)];
        if (!*f) *f = 1;
    }
}

// LFU_BATCH: one more batch for every distinct row of the last forward (rows
// of U are distinct, so plain increments suffice).
__global__ void __launch_bounds__(kBlock) k_plc_freq(DGlobal g, int64_t n) {
    if (*g.err) return;
    __shared__ int64_t s_start[RECMG_MAX_TABLES + 1];
    __shared__ int32_t s_uc[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_start[t] = g.tstart[t];
        if (t < g.T) s_uc[t] = g.st[t].ucount;
    }
    __syncthreads();
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int t = find_seg(s_start, g.T, i);
        if (i - s_start[t] < s_uc[t]) g.tabs[t].freq[g.U[i]] += 1;
    }
}

// Classify every distinct prefetch row of the fully associative tables (Alg.
// 1's prefetch loop taken as a set): resident -> flag the slot; missed by the
// last batch -> flag the miss; otherwise a new candidate, appended to NP.  One
// thread per slot of the prefetch index space; table t's distinct rows occupy
// [pstart[t], + pcount).  Set-associative tables play their prefetch rows as
// events in k_sa_place, which also counts the resident ones.
__global__ void __launch_bounds__(kBlock) k_plc_classify(DGlobal g, int32_t last_stamp, int64_t np) {
    if (*g.err) return;
    __shared__ int64_t s_pstart[RECMG_MAX_TABLES + 1];
    __shared__ int32_t s_pc[RECMG_MAX_TABLES];
    __shared__ int s_res[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_pstart[t] = g.pstart[t];
        if (t < g.T) {
            s_pc[t] = g.tabs[t].ways ? 0 : g.st[t].pcount;
            s_res[t] = 0;
        }
    }
    __syncthreads();
    const int stride_st = (int)(sizeof(TState) / 4);
    int64_t lo, hi;
    block_share(np, &lo, &hi);
    for (int64_t base = lo; base < hi; base += blockDim.x) {  // block-uniform
        const int64_t i = base + threadIdx.x;
        int t = 0;
        bool valid = false, isnew = false, resident = false;
        int32_t row = 0;
        if (i < hi) {
            t = find_seg(s_pstart, g.T, i);
            valid = i - s_pstart[t] < s_pc[t];
        }
        if (valid) {
            const DTable &tb = g.tabs[t];
            row = g.PU[i];
            const int32_t slot = find_slot(tb, row);
            if (slot >= 0) {
                // distinct prefetch rows name distinct slots: plain read-modify-write
                tb.slot_flags[slot] |= F_INP;
                resident = true;
                g.puref[i] = slot;
            } else {
                // distinct rows of the last batch carry its stamp in the rank word
                const uint32_t pos = bm_pos(tb, row);
                const uint4 rk = tb.rank[pos >> 5];
                const uint32_t bit = 1u << (pos & 31);
                if ((int32_t)rk.z == last_stamp && (rk.y & bit)) {
                    const int64_t ts = g.tstart[t];
                    const int32_t u = (int32_t)rk.x + __popc(rk.y & (bit - 1u));
                    const int64_t m = -(int64_t)g.slotU[ts + u] - 1;
                    g.mflags[ts + m] |= F_INP;  // distinct rows, distinct misses
                    g.puref[i] = ring_ref_miss((int32_t)m);
                } else {
                    isnew = true;
                }
            }
        }
        wave_count_lds(resident, t, s_res);  // counts only
        const int32_t k = wave_append(isnew, t, &g.st[0].npcount, stride_st);
        if (isnew) {
            g.NP[s_pstart[t] + k] = row;
            g.puref[i] = ring_ref_new(k);
        }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < g.T; t += blockDim.x)
        if (s_res[t]) atomicAdd(&g.st[t].p_res, s_res[t]);
}

// ----------------------------------------------------------------- ranking

__device__ __forceinline__ int pass_shift(const PlcParams &p, int pass) { return kRadixBits * (p.passes - 1 - pass); }
__device__ __forceinline__ int pass_width(const PlcParams &p, int pass) {
    return pass == 0 ? p.total_bits - kRadixBits * (p.passes - 1) : kRadixBits;
}

// Histogram increment, aggregated over the wave for the first active lane's
// bin: the keys of one table bunch up in few digits (LRU scores are batch
// numbers), and 64 lanes adding 1 to one LDS word would serialise.
__device__ __forceinline__ void hist_add(int *h, bool active, uint32_t bin) {
    const uint64_t act = __ballot(active);
    if (act == 0) return;
    const int lead = __ffsll((unsigned long long)act) - 1;
    const uint32_t b0 = (uint32_t)__shfl((int)bin, lead);
    const uint64_t same = __ballot(active && bin == b0);
    if ((int)(threadIdx.x & 63) == lead) atomicAdd(&h[b0], __popcll(same));
    if (active && bin != b0) atomicAdd(&h[bin], 1);
}

// Merge the block's histogram into the table's global one (non-zero bins).
// No fence and no "last block" here: on this GPU an agent-scope fence writes
// back the XCD's whole L2, and a histogram kernel has many blocks; the digit
// is picked by k_plc_pick after the kernel boundary instead.
__device__ __forceinline__ void hist_merge(const DGlobal &g, int t, const int *s_hist) {
    int *gh = g.hist + (int64_t)t * kRadix;
    for (int b = threadIdx.x; b < kRadix; b += blockDim.x)
        if (s_hist[b]) atomicAdd(&gh[b], s_hist[b]);
}

// The digit of one pass from a table's histogram in LDS: bins are taken from
// the top until `need` keys are covered; the bin reached (*digit) extends the
// threshold prefix and the keys still needed inside it (*rest) carry over to
// the next pass.  Every thread of the block calls; blockDim.x divides kRadix;
// the results are valid in every thread.
__device__ __forceinline__ void pick_digit(const int *s_hist, int need, int *tmp, int *digit, int *rest) {
    __shared__ int s_digit, s_rest;
    // thread k owns bin group (groups - 1 - k), so an exclusive scan gives the
    // keys in the groups above
    if (threadIdx.x == 0) {  // a histogram short of `need` (never, when the counts hold) keeps digit 0
        s_digit = 0;
        s_rest = need;
    }
    const int per = kRadix / (int)blockDim.x;
    const int grp = (int)blockDim.x - 1 - (int)threadIdx.x;
    int cs = 0;
    for (int b = 0; b < per; ++b) cs += s_hist[grp * per + b];
    int tot;
    const int above = block_excl_scan(cs, tmp, &tot);
    if (above < need && above + cs >= need) {
        int cum = above;
        for (int b = grp * per + per - 1; b >= grp * per; --b) {
            if (cum + s_hist[b] >= need) {
                s_digit = b;
                s_rest = need - cum;
                break;
            }
            cum += s_hist[b];
        }
    }
    __syncthreads();
    *digit = s_digit;
    *rest = s_rest;
    __syncthreads();
}

// One block per table: the digit of this pass from the table's global
// histogram (clearing it for the next pass).
__global__ void __launch_bounds__(kBlock) k_plc_pick(DGlobal g, PlcParams p, int pass) {
    if (*g.err) return;
    __shared__ int s_hist[kRadix];
    __shared__ int tmp[16];
    const int t = blockIdx.x;
    TState &st = g.st[t];
    if (g.tabs[t].ring_cap || st.sel_mode != SEL_SELECT) return;  // uniform over the block
    int *gh = g.hist + (int64_t)t * kRadix;
    for (int b = threadIdx.x; b < kRadix; b += blockDim.x) {
        s_hist[b] = gh[b];
        gh[b] = 0;
    }
    __syncthreads();
    const int need = pass == 0 ? table_counts(g.tabs[t], st, p).keep : st.need;
    int digit, rest;
    pick_digit(s_hist, need, tmp, &digit, &rest);
    if (threadIdx.x == 0) {
        st.prefix = pass == 0 ? (uint64_t)digit : ((st.prefix << kRadixBits) | (uint64_t)digit);
        st.need = rest;
    }
}

// The scans over every slot (score update, select passes, evict) take four
// consecutive slots per thread with 16-byte loads issued together: with one
// slot per thread and a score load that waited for the row load, they were
// bound by load latency (configuration 4's 78 million slots: about 1 TB/s).
// Slots [k0, k0 + 4) of a table, absent ones (k >= cap) reading row -1.
__device__ __forceinline__ void slot_quad(const int32_t *a, int64_t k0, int64_t cap, int32_t fill, int32_t (&v)[4]) {
    if (k0 + 3 < cap) {
        const uint4 w = gload16(a + k0);
        v[0] = (int32_t)w.x, v[1] = (int32_t)w.y, v[2] = (int32_t)w.z, v[3] = (int32_t)w.w;
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = k0 + i < cap ? (int32_t)gload4(a + k0 + i) : fill;
    }
}

// Scores of every candidate of table t (written back) and, when `sel`, the
// histogram of the first select pass, over items tid, tid + stride, ...
// (stride a multiple of 64: hist_add is wave-wide).
__device__ __forceinline__ void update_items(const DGlobal &g, const PlcParams &p, const DTable &tb, const Counts &c,
                                             int t, int *s_hist, bool sel, int64_t tid, int64_t stride) {
    const int64_t ts = g.tstart[t], ps = g.pstart[t];
    const int shift = pass_shift(p, 0);
    const uint32_t dmask = (1u << pass_width(p, 0)) - 1u;
    const int64_t cap = c.cap;
    // resident slots, four per thread; every lane runs the same number of
    // iterations (hist_add is wave-wide)
    const int64_t ngrp = (cap + 3) / 4, ngrp_r = (ngrp + 63) & ~(int64_t)63;
    for (int64_t q = tid; q < ngrp_r; q += stride) {
        const int64_t k0 = 4 * q;
        const int64_t lim = q < ngrp ? cap : 0;  // lanes past the last group see no slot
        int32_t row[4], sc[4], fl[4], tch[4];
        slot_quad(tb.slot_row, k0, lim, -1, row);
        slot_quad(tb.slot_score, k0, lim, 0, sc);
        slot_quad(reinterpret_cast<const int32_t *>(tb.slot_flags), k0, lim, 0, fl);
        slot_quad(tb.slot_touch, k0, lim, -1, tch);
        uint32_t cbw = 0;
        if (k0 + 3 < lim) cbw = gload4(tb.slot_cbit + k0);
        else
            for (int i = 0; i < 4; ++i)
                if (k0 + i < lim) cbw |= (uint32_t)tb.slot_cbit[k0 + i] << (8 * i);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t k = k0 + i;
            const int32_t r = row[i];
            int32_t s = sc[i];
            uint32_t f = (uint32_t)fl[i];
            const int cb = (int)((cbw >> (8 * i)) & 0xffu);
            if (k < lim) {
                if (p.prio) s = s > 0 ? s - 1 : 0;
                if (r >= 0 && tch[i] == p.last_stamp) {
                    f &= ~F_PF;
                    s = touch_score(p, tb, r, cb);
                }
                if ((f & F_INP) && s < p.pscore) s = p.pscore;
                // written back only where they change (most slots keep both)
                if (r >= 0 && s != sc[i]) tb.slot_score[k] = s;
                if (r >= 0 && (f & ~F_INP) != (uint32_t)fl[i]) tb.slot_flags[k] = f & ~F_INP;
            }
            if (sel) hist_add(s_hist, k < lim && r >= 0, (uint32_t)(make_key(s, r < 0 ? 0 : r, p.rowbits) >> shift) & dmask);
        }
        if (cbw) {  // caching bits are zero between placements
            if (k0 + 3 < lim) *reinterpret_cast<uint32_t *>(tb.slot_cbit + k0) = 0u;
            else
                for (int i = 0; i < 4; ++i)
                    if (k0 + i < lim && ((cbw >> (8 * i)) & 0xffu)) tb.slot_cbit[k0 + i] = 0;
        }
    }
    // candidates: the last batch's misses, then new prefetch rows
    const int64_t nc = (int64_t)c.nm + c.nnp, nc_r = (nc + 63) & ~(int64_t)63;
    for (int64_t k = tid; k < nc_r; k += stride) {
        int32_t row = -1, s = 0;
        if (k >= nc) {
        } else if (k < c.nm) {
            const int64_t m = ts + k;
            row = g.M[m];
            const uint32_t f = g.mflags[m];
            s = touch_score(p, tb, row, g.mcbit[m]);
            if ((f & F_INP) && s < p.pscore) s = p.pscore;
            g.mscore[m] = s;
        } else {
            row = g.NP[ps + (k - c.nm)];
            s = new_prefetch_score(p, tb, row);
        }
        if (sel) hist_add(s_hist, row >= 0, (uint32_t)(make_key(s, row < 0 ? 0 : row, p.rowbits) >> shift) & dmask);
    }
}

// Scores of every candidate (written back) and the first select pass.
__global__ void __launch_bounds__(kBlock) k_plc_update(DGlobal g, PlcParams p) {
    if (*g.err) return;
    __shared__ int s_hist[kRadix];
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    TState &st = g.st[t];
    if (tb.ring_cap) return;  // ranked in ring.hip
    const Counts c = table_counts(tb, st, p);
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        st.sel_mode = tb.ways ? SEL_NONE : c.mode;  // set-associative tables place in setassoc.hip
        st.plc_nm = c.nm;
    }
    if (tb.ways) return;
    const bool sel = c.mode == SEL_SELECT;
    if (sel)
        for (int b = threadIdx.x; b < kRadix; b += blockDim.x) s_hist[b] = 0;
    __syncthreads();
    update_items(g, p, tb, c, t, s_hist, sel, (int64_t)blockIdx.x * blockDim.x + threadIdx.x,
                 (int64_t)gridDim.x * blockDim.x);
    __syncthreads();
    if (sel) hist_merge(g, t, s_hist);
}

// Key of candidate k (k < nm: a miss of the last batch; else a new prefetch row).
__device__ __forceinline__ uint64_t cand_key(const DGlobal &g, const DTable &tb, const Counts &c, const PlcParams &p,
                                             int64_t ts, int64_t ps, int64_t k) {
    int32_t row, s;
    if (k < c.nm) {
        const int64_t m = ts + k;
        row = g.M[m];
        s = g.mscore[m];
    } else {
        row = g.NP[ps + (k - c.nm)];
        s = new_prefetch_score(p, tb, row);
    }
    return make_key(s, row, p.rowbits);
}

// Histogram of pass `pass` over the keys of table t whose higher digits equal
// `prefix`, over items tid, tid + stride, ... (stride a multiple of 64).
__device__ __forceinline__ void select_items(const DGlobal &g, const PlcParams &p, const DTable &tb, const Counts &c,
                                             int t, int *s_hist, int pass, uint64_t prefix, int64_t tid,
                                             int64_t stride) {
    const int64_t ts = g.tstart[t], ps = g.pstart[t];
    const int shift = pass_shift(p, pass);
    const int64_t cap = c.cap;
    const int64_t ngrp = (cap + 3) / 4, ngrp_r = (ngrp + 63) & ~(int64_t)63;
    for (int64_t q = tid; q < ngrp_r; q += stride) {
        const int64_t k0 = 4 * q;
        const int64_t lim = q < ngrp ? cap : 0;
        int32_t row[4], sc[4];
        slot_quad(tb.slot_row, k0, lim, -1, row);
        slot_quad(tb.slot_score, k0, lim, 0, sc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint64_t key = make_key(sc[i], row[i] < 0 ? 0 : row[i], p.rowbits);
            const bool in = row[i] >= 0 && (key >> (shift + kRadixBits)) == prefix;
            hist_add(s_hist, in, (uint32_t)(key >> shift) & (kRadix - 1));
        }
    }
    const int64_t nc = (int64_t)c.nm + c.nnp, nc_r = (nc + 63) & ~(int64_t)63;
    for (int64_t k = tid; k < nc_r; k += stride) {
        const uint64_t key = k < nc ? cand_key(g, tb, c, p, ts, ps, k) : 0;
        const bool in = k < nc && (key >> (shift + kRadixBits)) == prefix;
        hist_add(s_hist, in, (uint32_t)(key >> shift) & (kRadix - 1));
    }
}

__global__ void __launch_bounds__(kBlock) k_plc_select(DGlobal g, PlcParams p, int pass) {
    if (*g.err) return;
    __shared__ int s_hist[kRadix];
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    TState &st = g.st[t];
    if (tb.ring_cap || st.sel_mode != SEL_SELECT) return;  // uniform over the table's blocks
    const Counts c = table_counts(tb, st, p);
    for (int b = threadIdx.x; b < kRadix; b += blockDim.x) s_hist[b] = 0;
    __syncthreads();
    select_items(g, p, tb, c, t, s_hist, pass, st.prefix, (int64_t)blockIdx.x * blockDim.x + threadIdx.x,
                 (int64_t)gridDim.x * blockDim.x);
    __syncthreads();
    hist_merge(g, t, s_hist);
}

// Small tables: the whole ranking of a table in one block (scores, then every
// pass's histogram in LDS and its digit), one launch instead of 2 per pass.
constexpr int kRankSmallThreads = 1024;
__global__ void __launch_bounds__(kRankSmallThreads) k_plc_rank_small(DGlobal g, PlcParams p) {
    if (*g.err) return;
    __shared__ int s_hist[kRadix];
    __shared__ int tmp[16];
    const int t = blockIdx.x;
    const DTable &tb = g.tabs[t];
    TState &st = g.st[t];
    if (tb.ring_cap) return;
    const Counts c = table_counts(tb, st, p);
    if (threadIdx.x == 0) {
        st.sel_mode = tb.ways ? SEL_NONE : c.mode;
        st.plc_nm = c.nm;
    }
    if (tb.ways) return;
    const bool sel = c.mode == SEL_SELECT;
    for (int b = threadIdx.x; b < kRadix; b += blockDim.x) s_hist[b] = 0;
    __syncthreads();
    update_items(g, p, tb, c, t, s_hist, sel, threadIdx.x, blockDim.x);
    __syncthreads();  // also makes the scores written above visible to the block
    if (!sel) return;
    uint64_t prefix = 0;
    int need = c.keep;
    for (int pass = 0; pass < p.passes; ++pass) {
        if (pass > 0) {
            for (int b = threadIdx.x; b < kRadix; b += blockDim.x) s_hist[b] = 0;
            __syncthreads();
            select_items(g, p, tb, c, t, s_hist, pass, prefix, threadIdx.x, blockDim.x);
            __syncthreads();
        }
        int digit, rest;
        pick_digit(s_hist, need, tmp, &digit, &rest);
        prefix = pass == 0 ? (uint64_t)digit : ((prefix << kRadixBits) | (uint64_t)digit);
        need = rest;
    }
    if (threadIdx.x == 0) {
        st.prefix = prefix;
        st.need = need;
    }
}

// ----------------------------------------------------------------- evict / admit

// Slots a block collects in LDS before it reserves free-stack space for
// them: one atomic on the table's stack top per block in the common case (a
// few hundred evictions per block), instead of one per 256 slots scanned (a
// full cache of 19.5 million slots would queue some 76,000 of those on one
// word per table).  Freed slots enter the stack in no fixed order; slot
// numbers are not observable.
constexpr int kEvictBuf = 2048;

__global__ void __launch_bounds__(kBlock) k_plc_evict(DGlobal g, PlcParams p) {
    if (block_err(g)) return;
    __shared__ int tmp[16];
    __shared__ int s_base, s_n;
    __shared__ int32_t s_free[kEvictBuf];
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (tb.ways || tb.ring_cap) return;
    TState &st = g.st[t];
    const int mode = st.sel_mode;
    const uint64_t thr = st.prefix;
    const int lane = threadIdx.x & 63;
    if (threadIdx.x == 0) s_n = 0;
    __syncthreads();
    // reserve stack space for the collected slots with one atomic and write
    // them out; every thread calls (s_n is read after a barrier)
    auto flush = [&]() {
        const int n = s_n;
        if (n == 0) return;
        if (threadIdx.x == 0) s_base = atomicAdd(&st.free_top, n);
        __syncthreads();
        for (int i = threadIdx.x; i < n; i += blockDim.x) {
            const int64_t at = (int64_t)s_base + i;
            if (at < tb.cap) tb.free_stack[at] = s_free[i];
            else atomicOr(g.err, ERR_INTERNAL);
        }
        __syncthreads();
        if (threadIdx.x == 0) s_n = 0;
        __syncthreads();
    };
    int nev = 0;
    unsigned long long dig = 0;
    const int64_t cap = tb.cap;
    // four slots per thread; a block's iterations are uniform (its barriers)
    const int64_t ngrp = (cap + 3) / 4, stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t base = (int64_t)blockIdx.x * blockDim.x; base < ngrp; base += stride) {
        const int64_t q = base + threadIdx.x;
        const int64_t k0 = 4 * q;
        const int64_t lim = q < ngrp ? cap : 0;
        int32_t row[4], sc[4];
        slot_quad(tb.slot_row, k0, lim, -1, row);
        slot_quad(tb.slot_score, k0, lim, 0, sc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int64_t k = k0 + i;
            bool ev = false;
            if (row[i] >= 0) {
                if (kept(mode, make_key(sc[i], row[i], p.rowbits), thr)) {
                    dig += mix64(((unsigned long long)t << 40) | (unsigned long long)row[i]);
                } else {
                    ev = true;
                    map_delete(tb, row[i]);
                    tb.slot_row[k] = -1;
                    tb.slot_flags[k] = 0;
                }
            }
            // append the wave's freed slots to the block's list (one LDS atomic per wave)
            const uint64_t m = __ballot(ev);
            int wb = 0;
            if (lane == 0 && m) wb = atomicAdd(&s_n, __popcll(m));
            wb = __shfl(wb, 0);
            if (ev) s_free[wb + __popcll(m & ((1ull << lane) - 1ull))] = (int32_t)k;
            nev += ev ? 1 : 0;
        }
        __syncthreads();
        if (s_n > kEvictBuf - 4 * (int)blockDim.x) flush();  // room for one more pass of the block
    }
    __syncthreads();
    flush();
    const int e = block_sum(nev, tmp);
    const unsigned long long d = wave_sum64(dig);
    if ((threadIdx.x & 63) == 0 && d) atomicAdd(&st.digest_acc, d);
    if (threadIdx.x == 0 && e) {
        atomicAdd(&st.evicted, e);
        atomicAdd(&st.tomb, e);
    }
}

// Rebuild the map when deleted entries exceed 1/4 of it: clear it here and
// re-insert the surviving residents in k_map_refill.
__global__ void __launch_bounds__(kBlock) k_map_clear(DGlobal g) {
    if (*g.err) return;
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (tb.ways) return;
    TState &st = g.st[t];
    const int64_t mcap = (int64_t)tb.map_mask + 1;
    if ((int64_t)st.tomb * 4 <= mcap) return;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < mcap; i += (int64_t)gridDim.x * blockDim.x)
        tb.map[i] = make_int2(kEmpty, -1);
    if (blockIdx.x == 0 && threadIdx.x == 0) st.rebuild = 1;
}

__global__ void __launch_bounds__(kBlock) k_map_refill(DGlobal g) {
    if (*g.err) return;
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (tb.ways) return;
    TState &st = g.st[t];
    if (!st.rebuild) return;
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < tb.cap; k += (int64_t)gridDim.x * blockDim.x) {
        const int32_t row = tb.slot_row[k];
        if (row >= 0) map_insert(tb, row, (int32_t)k);
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st.tomb = 0;
}

__global__ void __launch_bounds__(kBlock) k_plc_admit(DGlobal g, PlcParams p) {
    if (block_err(g)) return;
    __shared__ int tmp[16];
    __shared__ int s_base;
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (tb.ways) return;
    TState &st = g.st[t];
    const Counts c = table_counts(tb, st, p);
    const int mode = st.sel_mode;
    const uint64_t thr = st.prefix;
    const int32_t top = st.free_top;
    const int64_t ts = g.ftstart[t], ps = g.pstart[t];
    const int64_t items = (int64_t)c.nm + c.nnp;
    int n_adm_miss = 0, n_fill = 0, n_pdrop = 0, n_mdrop = 0, n_reuse = 0;
    unsigned long long dig = 0;
    for (int64_t base = (int64_t)blockIdx.x * blockDim.x; base < items; base += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = base + threadIdx.x;
        int adm = 0;
        int32_t row = 0, s = 0;
        bool is_miss = false, inp = false;
        if (k < items) {
            is_miss = k < c.nm;
            if (is_miss) {
                row = g.M[ts + k];
                s = g.mscore[ts + k];
                inp = (g.mflags[ts + k] & F_INP) != 0;
            } else {
                row = g.NP[ps + (k - c.nm)];
                s = new_prefetch_score(p, tb, row);
                inp = true;
            }
            adm = kept(mode, make_key(s, row, p.rowbits), thr) ? 1 : 0;
        }
        int tot;
        const int ex = block_excl_scan(adm, tmp, &tot);
        if (threadIdx.x == 0 && tot) s_base = atomicAdd(&st.popped, tot);
        __syncthreads();
        if (k < items) {
            int32_t slot = -1;
            const int64_t fi = (int64_t)top - 1 - (s_base + ex);
            const int64_t fj = ts + ps + (s_base + ex);  // this row's entry in the fill list
            if (adm && (fi < 0 || fi >= tb.cap || (uint32_t)tb.free_stack[fi] >= (uint32_t)tb.cap || fj < 0 ||
                        fj >= g.fill_cap)) {
                atomicOr(g.err, ERR_INTERNAL);
                adm = 0;
            }
            if (adm) {
                slot = tb.free_stack[fi];
                tb.slot_row[slot] = row;
                tb.slot_score[slot] = s;
                tb.slot_flags[slot] = inp ? F_PF : 0u;
                tb.slot_touch[slot] = -1;
                n_reuse += map_insert(tb, row, slot);
                // the fill list: admitted row j of this table, its source and
                // slot: a miss's staging row; a prefetch row's host row, or for
                // a STAGED table the staged row of its candidate (the host
                // gathered NP[ps + i] into row ps + i)
                g.fill_src[fj] = is_miss ? (int32_t)k : tb.staged ? -(int32_t)(ps + (k - c.nm)) - 1 : -(row + 1);
                g.fill_slot[fj] = slot;
                if (tb.ring_cap) {  // where ring.hip finds the admitted rows' slots
                    if (is_miss) g.mslot[ts + k] = slot;
                    else g.npslot[ps + (k - c.nm)] = slot;
                }
                dig += mix64(((unsigned long long)t << 40) | (unsigned long long)row);
                if (is_miss) ++n_adm_miss;
                else ++n_fill;
            } else {
                if (is_miss) ++n_mdrop;
                if (inp) ++n_pdrop;
            }
        }
        __syncthreads();
    }
    const int a = block_sum(n_adm_miss, tmp), f = block_sum(n_fill, tmp);
    const int pd = block_sum(n_pdrop, tmp), md = block_sum(n_mdrop, tmp), ru = block_sum(n_reuse, tmp);
    const unsigned long long d = wave_sum64(dig);
    if ((threadIdx.x & 63) == 0 && d) atomicAdd(&st.digest_acc, d);
    if (threadIdx.x == 0) {
        if (a) atomicAdd(&st.adm_miss, a);
        if (f) atomicAdd(&st.p_fill, f);
        if (pd) atomicAdd(&st.p_drop, pd);
        if (md) atomicAdd(&st.m_drop, md);
        if (ru) atomicSub(&st.tomb, ru);
    }
}

// Copy admitted rows into their slots: misses from HBM staging, prefetch
// fills from pinned host memory over the host link (ZERO_COPY tables) or from
// rows the host staged and copied in (STAGED tables).  One launch per miss
// mode present (phase): the zero-copy tables' at once, the STAGED tables'
// after the host has staged their rows.  May run on a side stream,
// concurrently with the next forward and with the next placement: it reads
// only its own placement's fill list and descriptor (both double-buffered, see
// k_plc_finalize) and the staging buffer of the forward before that placement,
// which the next forward does not use.
__global__ void __launch_bounds__(kBlock) k_plc_fill(DGlobal g, const int64_t *__restrict__ fdesc, int phase) {
    if (*g.err) return;
    // the blocks that copy: zero-copy fills as many as k_plc_finalize chose
    // (fdesc[3]), HBM-to-HBM copies of STAGED rows the whole grid
    const int64_t nb = phase == FILL_STAGED ? (int64_t)gridDim.x
                       : fdesc[3] < 1 ? 1 : fdesc[3] > (int64_t)gridDim.x ? (int64_t)gridDim.x : fdesc[3];
    if ((int64_t)blockIdx.x >= nb) return;  // block-uniform
    __shared__ int32_t s_cnt[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t < g.T; t += blockDim.x) {
        const int64_t base = fdesc[4 * t], n = fdesc[4 * t + 1];
        const bool mine = (g.tabs[t].staged != 0) == (phase == FILL_STAGED);
        // admit wrote entries [base, base + n) and checked them against fill_cap
        s_cnt[t] = (mine && base >= 0 && n >= 0 && base + n <= g.fill_cap) ? (int32_t)n : 0;
    }
    __syncthreads();
    // entries were checked where admit and the set-associative placement wrote them
    copy_flat(
        g, s_cnt, nb,
        [&](int t, const DTable &tb, int64_t j) -> const char * {
            const int32_t src = g.fill_src[fdesc[4 * t] + j];
            if (src >= 0) return g.staging + (fdesc[4 * t + 2] + src) * g.stage_stride;  // admitted miss
            return tb.staged ? g.fstage + (int64_t)(-src - 1) * g.stage_stride  // prefetch row, host-staged
                             : tb.host + (int64_t)(-src - 1) * tb.row_bytes;    // prefetch row, zero-copy
        },
        [&](int t, const DTable &tb, int64_t j) { return tb.pool + (int64_t)g.fill_slot[fdesc[4 * t] + j] * tb.row_bytes; });
}

#ifndef RECMG_FILL_BLOCKS
#define RECMG_FILL_BLOCKS 112  // zero-copy fill alone on the host link
#endif
#ifndef RECMG_FILL_BLOCKS_SHARED
#define RECMG_FILL_BLOCKS_SHARED 256  // zero-copy fill beside the next forward's on-demand fetch
#endif
#ifndef RECMG_FILL_BLOCKS_BIG
#define RECMG_FILL_BLOCKS_BIG 512  // zero-copy fill beside a fetch of hundreds of MB
#endif
constexpr int kStagedFillBlocks = 1024;
// on-demand fetch bytes above which the next fetch is taken to share the link
// with the fill (below it, the fetch takes a few microseconds of link time)
constexpr unsigned long long kSharedFetchBytes = 1ull << 20;
// ... and above which the two hold the link together for tens of milliseconds
constexpr unsigned long long kBigFetchBytes = 1ull << 28;
constexpr int kFillGridBlocks = RECMG_FILL_BLOCKS > RECMG_FILL_BLOCKS_SHARED
                                    ? (RECMG_FILL_BLOCKS > RECMG_FILL_BLOCKS_BIG ? RECMG_FILL_BLOCKS : RECMG_FILL_BLOCKS_BIG)
                                    : (RECMG_FILL_BLOCKS_SHARED > RECMG_FILL_BLOCKS_BIG ? RECMG_FILL_BLOCKS_SHARED
                                                                                       : RECMG_FILL_BLOCKS_BIG);

// Publishes the counters and writes the fill descriptor of this placement
// (per table: first fill-list entry, entry count, base of its admitted misses
// in staging), which the fill reads instead of state the next placement resets.
// fdesc[3] (a spare word of table 0's entry) is the number of blocks the fill
// copies with: zero-copy fills take more when the last forward fetched at
// least 1 MB on demand, since the next forward's fetch will then share the
// host link (with fewer waves of its own the fill gets less of it), more
// still when it fetched at least 256 MB (the two then hold the link for tens
// of milliseconds, and the kernels beside them are a small part of the step),
// and fewer when the fill has the link to itself, so that it takes no more
// CUs than it needs from the kernels beside it.
// log_slot >= 0: the counters also go to that call's record of the stats log
// (the forward group of the record stays zero).
__global__ void k_plc_finalize(DGlobal g, int64_t *fdesc, int64_t log_slot) {
    if (*g.err) return;  // one block; nothing sets the word while it runs
    __shared__ unsigned long long s_mbytes;  // bytes of the last forward's on-demand misses
    if (threadIdx.x == 0) s_mbytes = 0;
    __syncthreads();
    unsigned long long mb = 0;
    for (int t = threadIdx.x; t < g.T; t += blockDim.x)
        mb += (unsigned long long)(g.st[t].mcount > 0 ? g.st[t].mcount : 0) * (unsigned long long)g.tabs[t].row_bytes;
    if (mb) atomicAdd(&s_mbytes, mb);
    __syncthreads();
    if (threadIdx.x == 0)
        fdesc[3] = s_mbytes >= kBigFetchBytes      ? RECMG_FILL_BLOCKS_BIG
                   : s_mbytes >= kSharedFetchBytes ? RECMG_FILL_BLOCKS_SHARED
                                                   : RECMG_FILL_BLOCKS;
    for (int t = threadIdx.x; t < g.T; t += blockDim.x) {
        TState &st = g.st[t];
        const DTable &tb = g.tabs[t];
        fdesc[4 * t] = g.ftstart[t] + g.pstart[t];
        fdesc[4 * t + 1] = st.popped;
        fdesc[4 * t + 2] = g.ftstart[t];
        if (!tb.ways) {  // set-associative tables count residents as they place
            st.free_top -= st.popped;  // popped stays: the fill may still read it
            st.n_res = tb.cap - st.free_top;
        }
        if (tb.ring_cap) {  // the ring's new front and back, the new pending list
            if (st.r_compact) {  // the live entries moved to the front of the other buffer
                st.r_buf ^= 1;
                st.r_tail = 0;
                st.r_head = st.r_moved + st.z1_len;
                st.r_compact = 0;
            } else {
                st.r_tail = st.r_cut;
                st.r_head += st.z1_len;
            }
            st.pend_n = st.pcount;
            st.pend_off = g.pstart[t];
            if (st.r_valid + st.pend_keep != st.n_res || st.r_head > tb.ring_cap) atomicOr(g.err, ERR_INTERNAL);
        }
        st.rebuild = 0;
        int64_t v[kPlcStats];
        v[0] = st.evicted;
        v[1] = st.adm_miss;
        v[2] = st.p_fill;
        v[3] = st.p_res;
        v[4] = st.p_drop;
        v[5] = st.m_drop;
        v[6] = st.n_res;
        v[7] = (int64_t)st.p_fill * tb.row_bytes;
        v[8] = st.pcount;
        for (int k = 0; k < kPlcStats; ++k) {
            st.last[kFwdStats + k] = v[k];
            st.total[kFwdStats + k] += v[k];
        }
        st.digest = st.digest_acc;
        if (log_slot >= 0) {
            int64_t *rec = g.stat_log + (log_slot * g.T + t) * (kNumStats + 1);
            for (int k = 0; k < kNumStats; ++k) rec[k] = k < kFwdStats ? 0 : v[k - kFwdStats];
            rec[kNumStats] = (int64_t)st.digest_acc;
        }
    }
}

// Initial state: every slot free, the free stack handing out slot 0 first.
__global__ void __launch_bounds__(kBlock) k_init_state(DGlobal g) {
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    for (int64_t k = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; k < tb.cap; k += (int64_t)gridDim.x * blockDim.x)
        tb.free_stack[k] = tb.cap - 1 - (int32_t)k;
    if (blockIdx.x == 0 && threadIdx.x == 0) g.st[t].free_top = tb.cap;
}

// ----------------------------------------------------------------- launchers

static inline unsigned grid_for(int64_t n, int per_block, unsigned cap) {
    int64_t b = (n + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > (int64_t)cap) b = cap;
    return (unsigned)b;
}

void launch_plc_prep(const DGlobal &g, const int64_t *poff, int64_t np, int32_t have_fwd, hipStream_t s) {
    k_plc_prep<<<1, kBlock, 0, s>>>(g, poff, np, have_fwd);
}

void launch_plc_bits(const DGlobal &g, const uint8_t *bits, int64_t n_last, hipStream_t s) {
    if (n_last <= 0) return;
    k_plc_bits<<<grid_for(n_last, kBlock * 4, 16384), kBlock, 0, s>>>(g, bits, n_last);
}

void launch_plc_freq(const DGlobal &g, int64_t n_last, hipStream_t s) {
    if (n_last <= 0) return;
    k_plc_freq<<<grid_for(n_last, kBlock * 4, 8192), kBlock, 0, s>>>(g, n_last);
}

void launch_plc_classify(const DGlobal &g, int32_t last_stamp, int64_t np, hipStream_t s) {
    if (np <= 0) return;
    k_plc_classify<<<grid_for(np, kBlock, 8192), kBlock, 0, s>>>(g, last_stamp, np);
}

void launch_plc_rank(const DGlobal &g, const PlcParams &p, int64_t item_bound, hipStream_t s) {
    if (item_bound <= kRankSmallItems) {  // a table's slots and candidates fit one block's loop
        k_plc_rank_small<<<g.T, kRankSmallThreads, 0, s>>>(g, p);
        return;
    }
    // few blocks per table: each block merges its non-zero histogram bins
    // into global memory
#ifndef RECMG_RANK_IPT
#define RECMG_RANK_IPT 32
#endif
    const dim3 grid(grid_for(item_bound, kBlock * RECMG_RANK_IPT, 512), g.T);
    k_plc_update<<<grid, kBlock, 0, s>>>(g, p);
    k_plc_pick<<<g.T, kBlock, 0, s>>>(g, p, 0);
    for (int pass = 1; pass < p.passes; ++pass) {
        k_plc_select<<<grid, kBlock, 0, s>>>(g, p, pass);
        k_plc_pick<<<g.T, kBlock, 0, s>>>(g, p, pass);
    }
}

void launch_plc_evict(const DGlobal &g, const PlcParams &p, int32_t max_cap, hipStream_t s) {
    k_plc_evict<<<dim3(grid_for(max_cap, kBlock * 4, 2048), g.T), kBlock, 0, s>>>(g, p);
}

void launch_plc_admit(const DGlobal &g, const PlcParams &p, int32_t max_cap, int32_t max_map, int64_t cand_bound,
                      hipStream_t s) {
    k_map_clear<<<dim3(grid_for(max_map, kBlock * 8, 2048), g.T), kBlock, 0, s>>>(g);
    k_map_refill<<<dim3(grid_for(max_cap, kBlock * 4, 2048), g.T), kBlock, 0, s>>>(g);
    k_plc_admit<<<dim3(grid_for(cand_bound, kBlock * items_per_thread(cand_bound, 4), 2048), g.T), kBlock, 0, s>>>(g, p);
}

void launch_plc_fill(const DGlobal &g, const int64_t *fdesc, int phase, hipStream_t s, hipEvent_t ev0,
                     hipEvent_t ev1) {
    // Zero-copy fills read the host: about a hundred blocks of 4-deep 16-byte
    // loads keep the host link full (about 2 MB in flight) when the fill has
    // it to itself.  Host reads hold a CU's L1 miss slots for microseconds, so
    // a larger grid slows every kernel that shares its CUs: with 512 blocks the
    // next forward's dedup, running alongside, took 0.88 ms on configuration 2
    // instead of 0.28 ms.  Measured on configuration 2 (no on-demand misses):
    // 80-96 blocks leave the link short, 160 and more slow the placement that
    // runs beside the fill (192: -8% lookups/s).  On configuration 3 the fill
    // shares the link with the next forward's fetch of about 330,000 misses
    // (85 MB), and 256 blocks gave +4% (512: -6%).  On configuration 5 the
    // fetch moves about 750 MB per batch beside a 3.8 GB fill, and 512 blocks
    // gave +2.7% against 256 (768 and 1024: the same as 512).  The grid holds
    // the largest count; k_plc_finalize writes how many of its blocks copy.
    // STAGED fills copy within HBM and take a full grid.
    const int blocks = phase == FILL_STAGED ? kStagedFillBlocks : kFillGridBlocks;
    if (ev0 || ev1) hipExtLaunchKernelGGL(k_plc_fill, dim3(blocks), dim3(kBlock), 0, s, ev0, ev1, 0, g, fdesc, phase);
    else k_plc_fill<<<blocks, kBlock, 0, s>>>(g, fdesc, phase);
}

void launch_plc_finalize(const DGlobal &g, int64_t *fdesc, int64_t log_slot, hipStream_t s) {
    k_plc_finalize<<<1, kBlock, 0, s>>>(g, fdesc, log_slot);
}

void launch_init_state(const DGlobal &g, int32_t max_cap, hipStream_t s) {
    k_init_state<<<dim3(grid_for(max_cap, kBlock * 4, 2048), g.T), kBlock, 0, s>>>(g);
}

}  // namespace recmg
