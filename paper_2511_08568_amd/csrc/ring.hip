// Resident rings: the LRU_BATCH placement of fully associative tables (Alg. 1
// and Alg. 2 applied between batches, Sec. VI-B) without ranking every slot.
//
// Under LRU_BATCH a score is the number b of the placement that last touched
// the row (the last batch's rows take lru_touch = b) or named it in a
// prefetch list (pscore = b + 1).  Scores only grow, and a placement changes
// the scores of the rows it touches or names and of no other.  So each table
// keeps its residents sorted by key (score, row), the smallest first:
//
//   ring      one run per earlier placement, in placement order: the rows
//             that took that placement's touch score, ascending (scores < b)
//   pending   the rows the previous placement named (score b), ascending;
//             kept apart because placement b adds rows of the same score
//
// Placement b then, per table:
//   touch   the last batch's hits and the prefetch list's residents take
//           their new scores; their ring entries go stale (slot_pos = -1)
//   zones   Z1, the keys of score b in row order: the pending rows neither
//           touched nor named again, merged with the last batch's rows that
//           are not named (hits; misses as candidates).  Z2, the keys of score
//           b + 1, is the prefetch list itself (PU, ascending)
//   cut     with D = |K| - min(Cap, |K|) keys to drop: if the ring holds at
//           least D live entries, its first D go (the D smallest keys) and
//           every candidate stays; otherwise the whole ring goes and the
//           threshold key falls at rank D - |ring| of Z1, else of Z2
//   evict   the ring entries before the cut (and Z1/Z2 residents below the
//           threshold)
//   admit   every candidate at or above the threshold (placement.hip)
//   append  Z1's kept keys go to the back of the ring as one run (holes
//           where a key was dropped); Z2's kept rows become the pending list
//
// The cost is O(touched + named + evicted) per placement, not O(Cap): live
// entries per chunk of kRingChunk entries are counted, so the cut is found by
// reading chunk counts.  Stale entries stay until the front passes them;
// when an append would run past the end of the buffer, the live entries are
// first compacted, in order, into the other buffer.  The kept set is the one
// the radix-select placement keeps: the same keys, ties in score broken by row.
#include <algorithm>

#include "launch.h"

namespace recmg {

constexpr int kRingThreads = 1024;  // one-block-per-table kernels: one entry of a chunk per thread
static_assert(kRingThreads == kRingChunk, "the cut takes a chunk's entries one per thread");
constexpr int kRingEvictBuf = 2048;

__device__ __forceinline__ bool ring_live(const DTable &tb, int32_t slot, int32_t e) {
    return slot >= 0 && slot < tb.cap && tb.slot_pos[slot] == e;
}

// First index of a[0, n) (ascending) holding a value >= v, or > v if upper.
__device__ __forceinline__ int32_t ring_bound(const int32_t *a, int32_t n, int32_t v, bool upper) {
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        const int32_t mid = (int32_t)(((uint32_t)lo + (uint32_t)hi) >> 1);
        const int32_t x = a[mid];
        if (x < v || (upper && x == v)) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// Table t's zone Z1: entries [pend_off + tstart[t], + z1_len) of g.zone.
// Tables' regions are disjoint: pend_off and tstart partition the prefetch
// and index spaces, and z1_len = pend_n + (last forward's distinct rows).
__device__ __forceinline__ int2 *ring_zone(const DGlobal &g, const TState &st, int t) {
    return g.zone + st.pend_off + g.tstart[t];
}

// One pass over the pending rows, the last batch's distinct rows and the
// prefetch list:
//  * Z1 by merging two ascending lists: pending entry i lands at i + (U rows
//    below it), U entry u at u + (pending rows at or below it), so a row in
//    both (a pending row the batch touched) takes two places, the pending one
//    a hole.  A key is a pending row neither touched nor named again, a hit or
//    miss the list does not name (F_INP, set by classification).
//  * new scores: hits take the touch score, or pscore if the list names them
//    (and lose F_PF); the list's untouched residents take pscore.  Their ring
//    entries go stale (slot_pos = -1).  F_INP stays until the append.
//  * the misses' scores, which admission reads.
// A thread reads a pending row's flags only if the batch did not touch it,
// and only hit threads write flags (of touched slots), so the reads see
// settled values.
__global__ void __launch_bounds__(kBlock) k_ring_touch(DGlobal g, PlcParams p) {
    if (*g.err) return;
    __shared__ int tmp[16];
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (!tb.ring_cap) return;
    TState &st = g.st[t];
    const int64_t ts = g.tstart[t], ps = g.pstart[t];
    const int32_t nu = p.have_fwd ? st.ucount : 0, pn = st.pend_n;
    const int32_t *prow = g.pend_row[st.pend_buf] + st.pend_off;
    const int32_t *pslot = g.pend_slot[st.pend_buf] + st.pend_off;
    const int32_t *urow = g.U + ts;
    int32_t *rcnt = tb.rcnt[st.r_buf];
    int2 *z = ring_zone(g, st, t);
    const int32_t n1 = pn + nu, n = n1 + st.pcount;
    if (blockIdx.x == 0 && threadIdx.x == 0) st.z1_len = n1;
    int keys = 0, stale = 0;
    for (int32_t j = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x); j < n; j += (int32_t)(gridDim.x * blockDim.x)) {
        int32_t sl = -1, s = 0;  // a resident whose score changes, and its new score
        if (j < n1) {
            int32_t row, at, ref = kRingHole;
            if (j < pn) {
                row = prow[j];
                const int32_t q = pslot[j];
                at = j + ring_bound(urow, nu, row, false);
                if (q >= 0 && q < tb.cap && tb.slot_touch[q] != p.last_stamp && !(tb.slot_flags[q] & F_INP)) ref = q;
            } else {
                const int32_t u = j - pn;
                row = urow[u];
                const int32_t h = g.slotU[ts + u];
                at = u + ring_bound(prow, pn, row, true);
                if (h >= 0) {
                    const uint32_t f = tb.slot_flags[h];
                    const bool inp = (f & F_INP) != 0;
                    if (!inp) ref = h;
                    sl = h;
                    s = inp ? p.pscore : p.lru_touch;
                    if (f & F_PF) tb.slot_flags[h] = f & ~F_PF;
                } else {
                    const int32_t m = -h - 1;
                    const bool inp = (g.mflags[ts + m] & F_INP) != 0;
                    g.mscore[ts + m] = inp ? p.pscore : p.lru_touch;
                    if (!inp) ref = ring_ref_miss(m);
                }
            }
            z[at] = make_int2(ref, row);
            keys += ref != kRingHole ? 1 : 0;
        } else {
            const int32_t v = g.puref[ps + (j - n1)];
            if (v >= 0 && tb.slot_touch[v] != p.last_stamp) {  // touched: its hit entry scored it
                sl = v;
                s = p.pscore;
            }
        }
        if (sl >= 0) {
            tb.slot_score[sl] = s;
            const int32_t e = tb.slot_pos[sl];
            if (e >= 0) {  // pending rows have no ring entry
                tb.slot_pos[sl] = -1;
                atomicSub(&rcnt[e / kRingChunk], 1);
                ++stale;
            }
        }
    }
    const int k = block_sum(keys, tmp), ns = block_sum(stale, tmp);
    if (threadIdx.x == 0) {
        if (k) atomicAdd(&st.z1_keys, k);
        if (ns) atomicSub(&st.r_valid, ns);
    }
}

// One block per table: where the D keys to drop end.  Sets sel_mode and the
// threshold key (st.prefix) that admission applies to the candidates, the
// ring's cut, whether Z1/Z2 residents are evicted, and whether the live
// entries after the cut move to the front of the other buffer (when this
// placement's run would not fit behind them), with each chunk's first new
// index.
__global__ void __launch_bounds__(kRingThreads) k_ring_cut(DGlobal g, PlcParams p) {
    if (*g.err) return;
    __shared__ int tmp[16];
    __shared__ int32_t s_at, s_rest;
    const int t = blockIdx.x;
    const DTable &tb = g.tabs[t];
    if (!tb.ring_cap) return;
    TState &st = g.st[t];
    const Counts c = table_counts(tb, st, p);
    const int64_t nk = (int64_t)st.n_res + c.nm + c.nnp;
    const int64_t drop = nk - c.keep;
    const int32_t nold = st.r_valid, z1 = st.z1_keys, z2 = st.pcount;
    const int32_t head = st.r_head, tail = st.r_tail;
    const int32_t *ring = tb.ring[st.r_buf];
    const int32_t *rcnt = tb.rcnt[st.r_buf];
    const int32_t nch = (int32_t)(((int64_t)head + kRingChunk - 1) / kRingChunk);
    bool bad = nold < 0 || (int64_t)nold + z1 + z2 != nk;  // every key sits in the ring, Z1 or Z2
    int32_t mode = c.mode, cut = tail, zev = 0, cut_live = 0;  // cut_live: live entries of cut's chunk before it
    uint64_t thr = make_key(p.lru_touch, 0, p.rowbits);  // below every key of Z1 and Z2
    if (!bad && drop > 0 && drop <= nold) {
        // the drop-th live entry from the front: whole chunks by their counts,
        // then the entries of the chunk that reaches it
        mode = SEL_SELECT;
        int32_t need = (int32_t)drop, cc = -1;
        for (int32_t base = tail / kRingChunk; base < nch; base += kRingThreads) {
            const int32_t ch = base + (int32_t)threadIdx.x;
            const int v = ch < nch ? rcnt[ch] : 0;
            int tot;
            const int ex = block_excl_scan(v, tmp, &tot);
            if (need <= tot) {  // block-uniform
                if (ex < need && ex + v >= need) {
                    s_at = ch;
                    s_rest = need - ex;
                }
                __syncthreads();
                cc = s_at;
                need = s_rest;
                __syncthreads();  // read before s_at is reused below
                break;
            }
            need -= tot;
        }
        if (cc < 0) {
            bad = true;
        } else {
            const int32_t e = cc * kRingChunk + (int32_t)threadIdx.x;
            const bool live = e >= tail && e < head && ring_live(tb, ring[e], e);
            if (threadIdx.x == 0) s_at = -1;
            int tot;
            const int ex = block_excl_scan(live ? 1 : 0, tmp, &tot);  // its barriers order s_at's reset
            if (live && ex + 1 == need) s_at = e + 1;
            __syncthreads();
            cut = s_at;
            if (cut < 0) bad = true;
            else if (cut / kRingChunk == cc) cut_live = need;
        }
    } else if (!bad && drop > nold) {
        // the whole ring goes; the threshold is the key of rank r of Z1, or of
        // rank r - |Z1| of Z2 (every prefetch row is a key)
        cut = head;
        zev = 1;
        const int32_t r = (int32_t)(drop - nold);
        if (r < z1) {
            const int2 *z = ring_zone(g, st, t);
            const int32_t n = st.z1_len;
            int32_t want = r;
            if (threadIdx.x == 0) s_at = -1;
            __syncthreads();
            for (int32_t base = 0; base < n; base += kRingThreads) {
                const int32_t j = base + (int32_t)threadIdx.x;
                const int2 zr = j < n ? z[j] : make_int2(kRingHole, 0);
                const bool key = zr.x != kRingHole;
                int tot;
                const int ex = block_excl_scan(key ? 1 : 0, tmp, &tot);
                if (want < tot) {  // block-uniform
                    if (key && ex == want) s_at = zr.y;
                    __syncthreads();
                    break;
                }
                want -= tot;
            }
            if (s_at < 0) bad = true;
            thr = make_key(p.lru_touch, s_at < 0 ? 0 : s_at, p.rowbits);
            mode = SEL_SELECT;
        } else if (r - z1 < z2) {
            thr = make_key(p.pscore, g.PU[g.pstart[t] + (r - z1)], p.rowbits);
            mode = SEL_SELECT;
        } else {
            mode = SEL_NONE;
        }
    } else if (!bad) {
        mode = SEL_ALL;  // nothing to drop
    }
    const int32_t moved = bad ? 0 : (int32_t)(drop <= 0 ? nold : drop <= nold ? nold - drop : 0);
    const bool compact = (int64_t)head + st.z1_len > tb.ring_cap;
    if (compact && moved > 0) {
        // first new index of each chunk from cut's on: its live entries at or after the cut
        int32_t run = 0;
        const int32_t c0 = cut / kRingChunk;
        for (int32_t base = c0; base < nch; base += kRingThreads) {
            const int32_t ch = base + (int32_t)threadIdx.x;
            const int v = ch < nch ? rcnt[ch] - (ch == c0 ? cut_live : 0) : 0;
            int tot;
            const int ex = block_excl_scan(v, tmp, &tot);
            if (ch < nch) tb.roff[ch] = run + ex;
            run += tot;
        }
        if (run != moved) bad = true;
    }
    if (threadIdx.x == 0) {
        if (bad) atomicOr(g.err, ERR_INTERNAL);
        st.sel_mode = mode;
        st.prefix = thr;
        st.plc_nm = c.nm;
        st.r_cut = cut;
        st.r_zevict = zev;
        st.r_compact = compact ? 1 : 0;
        st.r_moved = moved;
    }
}

// Evict the live ring entries in [r_tail, r_cut) and, when the cut passed
// the whole ring, the Z1 and Z2 residents below the threshold.  When
// compacting, the live entries after the cut go, in order, to the front of
// the other buffer (whose chunk counts are set here; their slots learn their
// new index in the append, after every move has read the old ones).  A
// chunk per block iteration, one count update per chunk; freed slots gather
// in LDS and reach the free stack with one atomic per flush.
__global__ void __launch_bounds__(kBlock) k_ring_evict(DGlobal g, PlcParams p) {
    if (block_err(g)) return;
    __shared__ int tmp[16];
    __shared__ int s_base, s_n;
    __shared__ int32_t s_free[kRingEvictBuf];
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (!tb.ring_cap) return;
    TState &st = g.st[t];
    const int lane = threadIdx.x & 63;
    if (threadIdx.x == 0) s_n = 0;
    __syncthreads();
    auto flush = [&]() {  // every thread calls
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
    int nev = 0, nring = 0;
    unsigned long long dig = 0;
    // frees slot sl (when ev) and lists it; every lane of the wave calls
    auto evict = [&](bool ev, int32_t sl) {
        if (ev) {
            const int32_t row = tb.slot_row[sl];
            map_delete(tb, row);
            tb.slot_row[sl] = -1;
            tb.slot_flags[sl] = 0;
            tb.slot_pos[sl] = -1;
            dig += mix64(((unsigned long long)t << 40) | (unsigned long long)(uint32_t)row);
            ++nev;
        }
        const uint64_t m = __ballot(ev);
        int wb = 0;
        if (lane == 0 && m) wb = atomicAdd(&s_n, __popcll(m));
        wb = __shfl(wb, 0);
        if (ev) s_free[wb + __popcll(m & ((1ull << lane) - 1ull))] = sl;
    };
    const int32_t tail = st.r_tail, cut = st.r_cut, head = st.r_head, moved = st.r_moved;
    const bool compact = st.r_compact != 0;
    const int cur = st.r_buf;
    const int32_t *ring = tb.ring[cur];
    int32_t *dst = tb.ring[cur ^ 1];
    // chunks [tail's, hi): up to the cut's, or to the last live one when moving
    const int32_t hi = compact && moved > 0 ? (int32_t)(((int64_t)head + kRingChunk - 1) / kRingChunk)
                       : cut > tail          ? (cut - 1) / kRingChunk + 1
                                             : 0;
    for (int32_t ch = tail / kRingChunk + (int32_t)blockIdx.x; ch < hi; ch += (int32_t)gridDim.x) {
        const int32_t e0 = ch * kRingChunk + 4 * (int32_t)threadIdx.x;
        const uint4 v = gload16(ring + e0);
        const int32_t sl[4] = {(int32_t)v.x, (int32_t)v.y, (int32_t)v.z, (int32_t)v.w};
        bool mv[4];
        int here = 0, nmv = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int32_t e = e0 + i;
            const bool live = e >= tail && e < head && ring_live(tb, sl[i], e);
            const bool ev = live && e < cut;
            mv[i] = live && !ev && compact;
            evict(ev, sl[i]);
            here += ev ? 1 : 0;
            nmv += mv[i] ? 1 : 0;
        }
        int tot;
        const int ex = block_excl_scan(nmv, tmp, &tot);
        if (tot) {  // block-uniform; chunks with movers lie at or after the cut's
            int32_t at = tb.roff[ch] + ex;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (!mv[i]) continue;
                if (at < moved) dst[at++] = sl[i];
                else atomicOr(g.err, ERR_INTERNAL);  // counts and entries disagree (never expected)
            }
        }
        const int hn = block_sum(here, tmp);
        if (threadIdx.x == 0 && hn) atomicSub(&tb.rcnt[cur][ch], hn);
        nring += here;
        __syncthreads();
        if (s_n > kRingEvictBuf - 4 * (int)blockDim.x) flush();
    }
    if (compact) {  // the other buffer's chunk counts: [0, moved) live
        const int32_t nchunks = tb.ring_cap / kRingChunk;
        for (int32_t ch = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x); ch < nchunks; ch += (int32_t)(gridDim.x * blockDim.x)) {
            const int64_t left = (int64_t)moved - (int64_t)ch * kRingChunk;
            tb.rcnt[cur ^ 1][ch] = left <= 0 ? 0 : left >= kRingChunk ? kRingChunk : (int32_t)left;
        }
    }
    if (st.r_zevict) {
        const int mode = st.sel_mode;
        const uint64_t thr = st.prefix;
        const int2 *z = ring_zone(g, st, t);
        const int64_t ps = g.pstart[t];
        const int32_t n1 = st.z1_len, n = n1 + st.pcount;
        for (int32_t base = (int32_t)(blockIdx.x * blockDim.x); base < n; base += (int32_t)(gridDim.x * blockDim.x)) {
            const int32_t k = base + (int32_t)threadIdx.x;
            int32_t sl = -1;
            if (k < n1) {
                const int2 zr = z[k];
                if (zr.x >= 0 && !kept(mode, make_key(p.lru_touch, zr.y, p.rowbits), thr)) sl = zr.x;
            } else if (k < n) {
                const int32_t v = g.puref[ps + (k - n1)];
                if (v >= 0 && !kept(mode, make_key(p.pscore, g.PU[ps + (k - n1)], p.rowbits), thr)) sl = v;
            }
            evict(sl >= 0, sl);
            __syncthreads();
            if (s_n > kRingEvictBuf - (int)blockDim.x) flush();
        }
    }
    __syncthreads();
    flush();
    const int e = block_sum(nev, tmp), er = block_sum(nring, tmp);
    const unsigned long long d = wave_sum64(dig);
    if (lane == 0 && d) atomicAdd(&st.digest_acc, 0ull - d);
    if (threadIdx.x == 0) {
        if (e) {
            atomicAdd(&st.evicted, e);
            atomicAdd(&st.tomb, e);
        }
        if (er) atomicSub(&st.r_valid, er);
    }
}

// After admission: when compacting, the moved slots' new indices (every move
// has read the old ones); Z1's kept keys to ring entries [head, + z1_len) of
// the buffer that stays current (a chunk per block iteration); Z2's rows and
// their slots (-1 where not kept) to the pending list of buffer wr, the kept
// residents losing F_INP.  Admitted candidates' slots come from admission.
__global__ void __launch_bounds__(kBlock) k_ring_append(DGlobal g, PlcParams p, int wr) {
    if (*g.err) return;
    __shared__ int tmp[16];
    const int t = blockIdx.y;
    const DTable &tb = g.tabs[t];
    if (!tb.ring_cap) return;
    TState &st = g.st[t];
    const int mode = st.sel_mode;
    const uint64_t thr = st.prefix;
    const int64_t ts = g.tstart[t], ps = g.pstart[t];
    const bool compact = st.r_compact != 0;
    const int buf = compact ? st.r_buf ^ 1 : st.r_buf;
    const int32_t n1 = st.z1_len, head = compact ? st.r_moved : st.r_head;
    if ((int64_t)head + n1 > tb.ring_cap) {  // compaction made room; never expected
        if (threadIdx.x == 0) atomicOr(g.err, ERR_INTERNAL);
        return;
    }
    int32_t *ring = tb.ring[buf];
    if (compact) {
        for (int32_t k = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x); k < head; k += (int32_t)(gridDim.x * blockDim.x)) {
            const int32_t sl = ring[k];
            if (sl >= 0 && sl < tb.cap) tb.slot_pos[sl] = k;
            else atomicOr(g.err, ERR_INTERNAL);
        }
    }
    const int2 *z = ring_zone(g, st, t);
    if (n1 > 0) {
        const int32_t c1 = (head + n1 - 1) / kRingChunk;
        for (int32_t ch = head / kRingChunk + (int32_t)blockIdx.x; ch <= c1; ch += (int32_t)gridDim.x) {
            int add = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int32_t e = ch * kRingChunk + 4 * (int32_t)threadIdx.x + i;
                if (e < head || e >= head + n1) continue;
                const int2 zr = z[e - head];
                int32_t sl = kRingHole;
                if (zr.x != kRingHole && kept(mode, make_key(p.lru_touch, zr.y, p.rowbits), thr))
                    sl = zr.x >= 0 ? zr.x : g.mslot[ts + (-1 - zr.x)];
                if (sl != kRingHole && (sl < 0 || sl >= tb.cap)) {
                    atomicOr(g.err, ERR_INTERNAL);
                    sl = kRingHole;
                }
                ring[e] = sl;
                if (sl != kRingHole) {
                    tb.slot_pos[sl] = e;
                    ++add;
                }
            }
            const int an = block_sum(add, tmp);
            if (threadIdx.x == 0 && an) {
                atomicAdd(&tb.rcnt[buf][ch], an);
                atomicAdd(&st.r_valid, an);
            }
        }
    }
    int keepn = 0;
    int32_t *prow = g.pend_row[wr] + ps, *pslot = g.pend_slot[wr] + ps;
    for (int32_t i = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x); i < st.pcount; i += (int32_t)(gridDim.x * blockDim.x)) {
        const int32_t row = g.PU[ps + i], v = g.puref[ps + i];
        int32_t sl = -1;
        if (kept(mode, make_key(p.pscore, row, p.rowbits), thr)) {
            if (v >= 0) {
                sl = v;
                tb.slot_flags[v] &= ~F_INP;
            } else {
                sl = v > kRingNewBase ? g.mslot[ts + (-1 - v)] : g.npslot[ps + (kRingNewBase - v)];
            }
        }
        prow[i] = row;
        pslot[i] = sl;
        keepn += sl >= 0 ? 1 : 0;
    }
    const int kn = block_sum(keepn, tmp);
    if (threadIdx.x == 0 && kn) atomicAdd(&st.pend_keep, kn);
    if (blockIdx.x == 0 && threadIdx.x == 0) st.pend_buf = wr;
}

// ----------------------------------------------------------------- launchers

static inline unsigned ring_grid(int64_t n, int per_block, unsigned cap) {
    int64_t b = (n + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > (int64_t)cap) b = cap;
    return (unsigned)b;
}

void launch_ring_rank(const DGlobal &g, const PlcParams &p, int64_t item_bound, hipStream_t s) {
    k_ring_touch<<<dim3(ring_grid(item_bound, kBlock * items_per_thread(item_bound, 4), 1024), g.T), kBlock, 0, s>>>(g, p);
    k_ring_cut<<<g.T, kRingThreads, 0, s>>>(g, p);
}

void launch_ring_evict(const DGlobal &g, const PlcParams &p, int64_t item_bound, int32_t ring_chunks, hipStream_t s) {
    // the cut is typically a few chunks past the front; a compaction walks
    // every chunk, so blocks loop
    const unsigned gx = std::max(ring_grid(item_bound, kBlock * 4, 256), ring_grid(ring_chunks, 64, 256));
    k_ring_evict<<<dim3(gx, g.T), kBlock, 0, s>>>(g, p);
}

void launch_ring_store(const DGlobal &g, const PlcParams &p, int64_t item_bound, int32_t max_cap, int wr,
                       hipStream_t s) {
    const unsigned gx = std::max(ring_grid(item_bound, kBlock * 4, 1024), ring_grid(max_cap, kBlock * 16, 1024));
    k_ring_append<<<dim3(gx, g.T), kBlock, 0, s>>>(g, p, wr);
}

}  // namespace recmg
