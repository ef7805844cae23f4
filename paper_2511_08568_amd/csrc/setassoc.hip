// Placement in W-way set-associative tables: Alg. 1 (load_embeddings) and
// Alg. 2 (gpu_buffer_populate) of Sec. VI-B run literally inside each set.
//
// Row r lives in set r mod S, slots [set * W, + W).  Sets are independent, so
// one wave takes one set, lane w holding way w (row, score, flags) in
// registers, and plays the set's events in order:
//   A. rows the last batch touched (slot_touch = its stamp) lose their
//      prefetch flag and take the touch score: LRU_BATCH the batch stamp,
//      PRIORITY the OR of their caching bits + eviction_speed, LFU_BATCH the
//      row's batch count;
//   B. the set's misses of the last batch, ascending by row, are inserted with
//      their touch score;
//   C. the set's distinct prefetch rows, ascending by row: a resident one keeps
//      max(score, prefetch score), any other is inserted with the prefetch score
//      (LFU_BATCH: its batch count).
// Insert: the lowest free way, else Alg. 2 over the set: the victim is the
// lowest way holding the minimum score (scores before this scan), then under
// PRIORITY every way of the set ages by one, saturating at 0.
//
// The events of a set come from the dedup lists: U (the last forward's
// distinct rows) and PU (this placement's distinct prefetch rows) are emitted
// grouped by set and ascending within a set (bm_pos), so each set's events are
// two contiguous segments, found by k_sa_heads and kept in DTable::seg.
//
// A way whose row at the end differs from its row at the start gets a fill
// entry (misses of the last batch from HBM staging, every other row from the
// host) and the prefetch flag [row in P]; the fill itself is k_plc_fill's.
// Counters follow the set definitions: evicted |R \ R'|, admitted_miss
// |(R' \ R) ∩ M|, prefetch_fill = rows read from the host (new rows and rows
// moved to another way), prefetch_dropped |P \ (R ∪ R')|, miss_dropped
// |M \ R'|; the digest and the resident count change by what came and went.
#include <algorithm>

#include "launch.h"

namespace recmg {

// Segment bounds of every set that has events.  Index space: the last
// forward's distinct rows (all tables, nu), then this placement's distinct
// prefetch rows (np).  A first element of its set in its table's list writes
// the begin, a last element the end.  A prefetch row also gets its staging
// row if the last batch missed it (pfrom): found here, where every row is
// looked up in parallel, its two dependent loads stay off the sets' chains.
__global__ void __launch_bounds__(kBlock) k_sa_heads(DGlobal g, int64_t nu, int64_t np, int32_t have_fwd,
                                                     int32_t last_stamp) {
    if (*g.err) return;
    __shared__ int64_t s_ts[RECMG_MAX_TABLES + 1], s_ps[RECMG_MAX_TABLES + 1];
    __shared__ int32_t s_uc[RECMG_MAX_TABLES], s_pc[RECMG_MAX_TABLES];
    for (int t = threadIdx.x; t <= g.T; t += blockDim.x) {
        s_ts[t] = g.tstart[t];
        s_ps[t] = g.pstart[t];
        if (t < g.T) {
            s_uc[t] = have_fwd ? g.st[t].ucount : 0;
            s_pc[t] = g.st[t].pcount;
        }
    }
    __syncthreads();
    const int64_t n = nu + np;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const bool is_u = i < nu;
        const int64_t k = is_u ? i : i - nu;
        const int64_t *starts = is_u ? s_ts : s_ps;
        const int t = find_seg(starts, g.T, k);
        const DTable &tb = g.tabs[t];
        const int64_t loc = k - starts[t];
        const int32_t cnt = is_u ? s_uc[t] : s_pc[t];
        if (!tb.ways || loc >= cnt) continue;
        const int32_t *list = (is_u ? g.U : g.PU) + starts[t];
        const uint32_t ns = (uint32_t)tb.nsets;
        const uint32_t set = (uint32_t)list[loc] % ns;
        if (!is_u) {
            int32_t from = -1;
            if (have_fwd) {
                const int32_t r = list[loc];
                const uint32_t pos = bm_pos(tb, r);
                const uint4 rk = tb.rank[pos >> 5];
                const uint32_t bit = 1u << (pos & 31);
                if ((int32_t)rk.z == last_stamp && (rk.y & bit)) {
                    const int32_t su = g.slotU[s_ts[t] + (int32_t)rk.x + __popc(rk.y & (bit - 1u))];
                    if (su < 0) from = -su - 1;
                }
            }
            g.pfrom[starts[t] + loc] = from;
        }
        int *sg = reinterpret_cast<int *>(tb.seg + set);
        if (loc == 0 || (uint32_t)list[loc - 1] % ns != set) sg[is_u ? 0 : 2] = (int)loc;
        if (loc + 1 == cnt || (uint32_t)list[loc + 1] % ns != set) sg[is_u ? 1 : 3] = (int)(loc + 1);
    }
}

// Minimum of v over each group of HL lanes (HL = 64: the wave, 32: each
// half), returned per group as a scalar (m0 of lanes 0-31 or the wave, m1 of
// lanes 32-63): DPP within rows of 16 lanes, row broadcasts across rows, reads
// of the groups' last lanes.  Every lane must be active.
template <int HL>
__device__ __forceinline__ void group_min_dpp(int v, int &m0, int &m1) {
    v = min(v, __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
    v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
    v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false));  // row_half_mirror
    v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false));  // row_mirror
    v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x142, 0xA, 0xF, false));  // row_bcast:15 into rows 1, 3
    if constexpr (HL == 64) {
        v = min(v, __builtin_amdgcn_update_dpp(v, v, 0x143, 0xC, 0xF, false));  // row_bcast:31 into rows 2, 3
        m0 = m1 = __builtin_amdgcn_readlane(v, 63);
    } else {
        m0 = __builtin_amdgcn_readlane(v, 31);
        m1 = __builtin_amdgcn_readlane(v, 63);
    }
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// tot[k] for a lane-dependent k in [1, 7] (a select chain: no dynamic register indexing)
__device__ __forceinline__ int64_t pick_lane_tot(const int (&tot)[8], int k) {
    int v = tot[1];
#pragma unroll
    for (int i = 2; i < 8; ++i) v = k == i ? tot[i] : v;
    return v;
}

static_assert(kSaWaves == 16, "the block's counts are added up over one DPP row of 16 lanes");

// SPW sets per wave (2 for tables with many sets of W <= 32 ways, lanes
// 32h .. 32h + 31 taking set h; else 1), lane w of a set holding way w;
// kSaWaves * SPW sets per block.  The sets of a wave play their events side
// by side, one event of each per step, so a wave's chain of dependent loads
// serves two sets when the ways fit in half a wave; a step then costs more
// instructions, so tables with few sets (many events each, played one after
// another) keep one set per wave.  Blocks run table by table, tables with the
// fewest sets first: their sets take the most events each, and the longest
// waves should start first.  The counters and the fill-list space of a
// block's sets are added up by its first wave and taken with one atomic each
// per block (an atomic per set would queue hundreds of thousands of them on
// the same few words of a table with many sets).
template <int SPW>
__global__ void __launch_bounds__(kSaBlock) k_sa_place(DGlobal g, PlcParams p, int32_t nsa, int32_t boff) {
    constexpr int HL = 64 / SPW;  // lanes per set
    __shared__ int s_cnt[kSaWaves][8];
    __shared__ unsigned long long s_dig[kSaWaves];
    __shared__ int s_off[kSaWaves];
    // No early return: every wave reaches the block's barriers.  A wave that
    // finds the error word set (another block may set it meanwhile) does no work.
    const bool err = *g.err != 0;
    const int32_t bid = (int32_t)blockIdx.x + boff;  // block of the whole set-associative placement
    const int kt = find_seg32(g.sa_bstart, nsa, bid);
    const int t = g.sa_btab[kt];
    const DTable &tb = g.tabs[t];
    TState &st = g.st[t];
    const int W = tb.ways;
    const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int h = lane / HL, wl = lane % HL;  // this lane's set of the wave, and its way
    const bool hi = h != 0;
    // this lane's half of a 64-bit ballot (the whole ballot when SPW == 1)
    auto half = [&](uint64_t b) -> uint64_t { return SPW == 1 ? b : (hi ? b >> 32 : b & 0xffffffffull); };
    // value of lane k of this lane's set (k wave-uniform per set: k0 for set 0, k1 for set 1)
    auto pick = [&](int v, int k0, int k1) -> int {
        if constexpr (SPW == 1) return __builtin_amdgcn_readlane(v, k0);
        const int a = __builtin_amdgcn_readlane(v, k0 & 31), b = __builtin_amdgcn_readlane(v, 32 + (k1 & 31));
        return hi ? b : a;
    };
    const int64_t set = ((int64_t)(bid - g.sa_bstart[kt]) * kSaWaves + wid) * SPW + h;
    int4 sg = make_int4(0, 0, 0, 0);
    // the ways are read beside the segment bounds, before it is known whether
    // the set has events (about half of a large cache's sets have none in a
    // placement): one round trip less on every set's chain
    int32_t w_row = -1, w_score = 0, w_touch = -1, w_cbit = 0;
    uint32_t w_flags = 0;
    if (!err && set < tb.nsets) {
        const uint4 sv = gload16(tb.seg + set);
        sg = make_int4((int)sv.x, (int)sv.y, (int)sv.z, (int)sv.w);
        if (wl < W) {
            const int64_t sl = set * W + wl;
            w_row = (int32_t)gload4(tb.slot_row + sl);
            w_score = (int32_t)gload4(tb.slot_score + sl);
            w_flags = gload4(tb.slot_flags + sl);
            w_touch = (int32_t)gload4(tb.slot_touch + sl);
            // caching bits are set only under PRIORITY (zero otherwise)
            if (p.prio) w_cbit = RECMG_GLOBAL(uint8_t, tb.slot_cbit + sl);
        }
    }
    const bool active = sg.x != sg.y || sg.z != sg.w;  // uniform over the set's lanes
    const bool way = wl < W && active;
    const int64_t slot = set * W + wl;
    const int64_t pb = g.pstart[t];
    // per-set event counts, as scalars (set 1's are 0 when SPW == 1)
    auto both = [&](int v, int &v0, int &v1) {
        v0 = __builtin_amdgcn_readlane(v, 0);
        v1 = SPW == 1 ? 0 : __builtin_amdgcn_readlane(v, 32);
    };
    int nu0, nu1, np0, np1;
    both(sg.y - sg.x, nu0, nu1);
    both(sg.w - sg.z, np0, np1);
    // results of this lane's way, and of the wave
    int32_t row = -1, src = -1;
    bool changed = false, from_m = false;
    int c_ev = 0, c_am = 0, c_fill = 0, c_pd = 0, c_md = 0, c_res = 0, c_pres = 0;
    unsigned long long dsum = 0;
    if (ballot(active)) {
    if (active && wl == 0) tb.seg[set] = make_int4(0, 0, 0, 0);
    // A set's events are played one after another: a wave with many of them
    // is the kernel's critical path, so it takes issue slots first.
    if (max(nu0 + np0, nu1 + np1) > 256) __builtin_amdgcn_s_setprio(3);

    // The first chunk of each event list is loaded with the ways (one round
    // trip for all of them; most sets have fewer than HL events of each kind).
    const int64_t ub = g.tstart[t];
    int32_t u0_r = 0, u0_su = 0, p0_r = -1, p0_from = -1;
    if (sg.x + wl < sg.y) {
        u0_r = g.U[ub + sg.x + wl];
        u0_su = g.slotU[ub + sg.x + wl];
    }
    if (sg.z + wl < sg.w) {
        p0_r = g.PU[pb + sg.z + wl];
        p0_from = g.pfrom[pb + sg.z + wl];
    }

    // A. this set's ways; rows the last batch touched take the touch score
    int32_t row0 = -1, score = 0;
    uint32_t flags = 0;
    if (way) {
        row0 = w_row;
        score = w_score;
        flags = w_flags & F_PF;
        if (row0 >= 0 && w_touch == p.last_stamp) {
            const int cb = w_cbit;
            if (cb) tb.slot_cbit[slot] = 0;
            flags = 0;
            score = touch_score(p, tb, row0, cb);
        }
    }
    row = row0;        // src: this lane's last insertion, staging index of a miss or -1 (host)
    bool inp = false;  // this lane's row is named by the prefetch list

    // Insert row r with score v (from: its staging index, or -1) into this
    // lane's set when `act` (uniform over the set): the lowest free way, else
    // the lowest way holding the set's minimum score, after which, under
    // PRIORITY, every way of the set ages by one (saturating at 0).  Returns
    // the way taken.  Every lane of the wave calls.
    auto insert = [&](bool act, int32_t r, int32_t v, int32_t from) -> int {
        const uint64_t fr = half(ballot(way && row < 0));
        int m0, m1;
        group_min_dpp<HL>(way ? score : INT32_MAX, m0, m1);
        const int m = hi ? m1 : m0;
        const uint64_t mins = half(ballot(way && score == m));
        const int victim = __ffsll((unsigned long long)(fr ? fr : mins)) - 1;
        if (act) {
            if (!fr && p.prio && way) score = score > 0 ? score - 1 : 0;
            if (wl == victim) {
                row = r;
                score = v;
                src = from;
                inp = false;
            }
        }
        return victim;
    };

    // B. misses of the last batch, ascending.  Each chunk of HL distinct rows
    // of a set is loaded lane-parallel with the misses' touch scores, then
    // played one miss at a time from registers.
    int nmiss = 0;
    for (int32_t i0 = 0; i0 < max(nu0, nu1); i0 += HL) {
        const int32_t i = sg.x + i0 + wl;
        const bool in = i < sg.y;
        int32_t r = u0_r, su = u0_su, v = 0;
        if (in) {
            if (i0 > 0) {
                r = g.U[ub + i];
                su = g.slotU[ub + i];
            }
            if (su < 0) v = touch_score(p, tb, r, p.prio ? g.mcbit[ub + (-su - 1)] : 0);
        }
        const uint64_t mm = ballot(in && su < 0);
        nmiss += __popcll(mm);
        uint64_t mm0 = SPW == 1 ? mm : mm & 0xffffffffull, mm1 = SPW == 1 ? 0 : mm >> 32;
        while (mm0 | mm1) {
            const int j0 = mm0 ? __ffsll((unsigned long long)mm0) - 1 : 0;
            const int j1 = mm1 ? __ffsll((unsigned long long)mm1) - 1 : 0;
            const bool act = hi ? mm1 != 0 : mm0 != 0;
            insert(act, pick(r, j0, j1), pick(v, j0, j1), -pick(su, j0, j1) - 1);
            mm0 &= mm0 ? mm0 - 1 : 0;
            mm1 &= mm1 ? mm1 - 1 : 0;
        }
    }

    // C. distinct prefetch rows, ascending.  Each lane first finds whether its
    // row missed in the last batch (then it is still in staging).
    for (int32_t i0 = 0; i0 < max(np0, np1); i0 += HL) {
        const int32_t i = sg.z + i0 + wl;
        int32_t r = -1, from = -1, v = 0;
        if (i < sg.w) {
            r = i0 > 0 ? g.PU[pb + i] : p0_r;
            from = i0 > 0 ? g.pfrom[pb + i] : p0_from;  // staging row of a row the last batch missed (k_sa_heads)
            v = new_prefetch_score(p, tb, r);
        }
        const int c0 = min(HL, np0 - i0), c1 = min(HL, np1 - i0);
        for (int j = 0; j < max(c0, c1); ++j) {
            const bool act = j < (hi ? c1 : c0);
            const int32_t rr = pick(r, j, j);
            const uint64_t hit = half(ballot(way && row == rr));
            if (act && hit && wl == __ffsll((unsigned long long)hit) - 1) {
                if (score < p.pscore) score = p.pscore;
                inp = true;
            }
            const int w = insert(act && !hit, rr, pick(v, j, j), pick(from, j, j));
            if (act && !hit && wl == w) inp = true;
        }
    }

    // counters: compare the set's rows at the start and at the end.  A set's
    // rows are distinct at every point, so a row that left an unchanged way
    // can only be found in a changed one, and the search runs over those (a
    // row of one set never equals a row of another, so the search may run
    // over the changed ways of the whole wave).
    const uint64_t dm = ballot(way && row != row0);
    bool kept0 = (dm >> lane & 1ull) == 0, was = kept0;
    for (uint64_t m = dm; m; m &= m - 1) {
        const int k = __ffsll((unsigned long long)m) - 1;
        kept0 |= __builtin_amdgcn_readlane(row, k) == row0;
        was |= __builtin_amdgcn_readlane(row0, k) == row;
    }
    const bool evicted = way && row0 >= 0 && !kept0;
    changed = way && row >= 0 && row != row0;
    const bool fresh = way && row >= 0 && !was;  // in R' \ R
    from_m = changed && src >= 0;
    unsigned long long dig = 0;
    if (fresh) dig += mix64(((unsigned long long)t << 40) | (unsigned long long)row);
    if (evicted) dig -= mix64(((unsigned long long)t << 40) | (unsigned long long)row0);
    const int d_res = (way && row >= 0 ? 1 : 0) - (way && row0 >= 0 ? 1 : 0);

    // prefetch rows in R (prefetch_resident) and in neither R nor R'
    // (prefetch_dropped); R ∪ R' = the rows at the start and the rows of the
    // changed ways (again the whole wave may be searched)
    const uint64_t wm = ballot(way);
    int pdrop = 0, pres = 0;
    for (int32_t i0 = 0; i0 < max(np0, np1); i0 += HL) {
        const int32_t i = sg.z + i0 + wl;
        const int32_t r = i < sg.w ? (i0 == 0 ? p0_r : g.PU[pb + i]) : -1;  // the first chunk is in registers
        bool in_r = false, in = false;
        for (uint64_t m = wm; m; m &= m - 1) in_r |= __builtin_amdgcn_readlane(row0, __ffsll((unsigned long long)m) - 1) == r;
        for (uint64_t m = dm; m; m &= m - 1) in |= __builtin_amdgcn_readlane(row, __ffsll((unsigned long long)m) - 1) == r;
        pres += (i < sg.w && in_r) ? 1 : 0;
        pdrop += (i < sg.w && !in_r && !in) ? 1 : 0;
    }

    if (way) {
        tb.slot_row[slot] = row;
        tb.slot_score[slot] = score;
        tb.slot_flags[slot] = changed ? (inp ? F_PF : 0u) : flags;
        if (changed) tb.slot_touch[slot] = -1;
    }
    c_ev = wave_sum(evicted ? 1 : 0);
    c_am = wave_sum(from_m ? 1 : 0);
    c_fill = wave_sum(changed && !from_m ? 1 : 0);
    c_pd = wave_sum(pdrop);
    c_pres = wave_sum(pres);
    c_md = nmiss - c_am;
    c_res = wave_sum(d_res);
    dsum = wave_sum64(dig);
    }  // some set of the wave active

    // the block's totals: one atomic per counter, one for the fill-list space
    const uint64_t chm = ballot(changed);
    if (lane == 0) {
        s_cnt[wid][0] = __popcll(chm);
        s_cnt[wid][1] = c_ev;
        s_cnt[wid][2] = c_am;
        s_cnt[wid][3] = c_fill;
        s_cnt[wid][4] = c_pd;
        s_cnt[wid][5] = c_md;
        s_cnt[wid][6] = c_res;
        s_cnt[wid][7] = c_pres;
        s_dig[wid] = dsum;
    }
    __syncthreads();
    // Wave 0 adds them up, lane w holding wave w's counts: inclusive scans
    // over the 16 lanes of the first row by DPP row shifts (lanes past the row
    // edge read 0), the totals in lane 15.
    if (wid == 0) {
        auto row_scan = [&](int v) {
            v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, true);  // row_shr:1
            v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, true);  // row_shr:2
            v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, true);  // row_shr:4
            v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, true);  // row_shr:8
            return v;
        };
        const bool mine = lane < kSaWaves;
        const int c0 = mine ? s_cnt[lane][0] : 0;
        const int sc0 = row_scan(c0);
        const int tot0 = __builtin_amdgcn_readlane(sc0, kSaWaves - 1);
        int tot[8];
        tot[0] = tot0;
#pragma unroll
        for (int k = 1; k < 8; ++k) tot[k] = __builtin_amdgcn_readlane(row_scan(mine ? s_cnt[lane][k] : 0), kSaWaves - 1);
        const unsigned long long d = wave_sum64(mine ? s_dig[lane] : 0ull);
        int base = 0;
        if (lane == 0 && tot0) base = atomicAdd(&st.popped, tot0);
        base = __builtin_amdgcn_readfirstlane(base);
        if (mine) s_off[lane] = base + sc0 - c0;
        // the other counts go to this block's record (plain stores: atomics from
        // every block would queue on the table state's few lines), added up per
        // table by k_sa_sum
        if (lane < 7) g.sa_part[(int64_t)bid * 8 + lane] = pick_lane_tot(tot, lane + 1);
        if (lane == 7) g.sa_part[(int64_t)bid * 8 + 7] = (int64_t)d;  // the digest's bits
    }
    __syncthreads();
    if (changed) {
        const int64_t fj = g.ftstart[t] + pb + s_off[wid] + __popcll(chm & ((1ull << lane) - 1ull));
        if (fj < 0 || fj >= g.fill_cap) {
            atomicOr(g.err, ERR_INTERNAL);
        } else {
            g.fill_src[fj] = from_m ? src : -(row + 1);
            g.fill_slot[fj] = (int32_t)slot;
        }
    }
}

// The placement blocks' records added to their tables' counters: blockIdx.x
// is the table (in sa_btab order), blockIdx.y one of gridDim.y slices of its
// blocks; one atomic per counter per slice.
__global__ void __launch_bounds__(1024) k_sa_sum(DGlobal g, int32_t nsa) {
    if (*g.err) return;
    __shared__ long long tmp[16];
    __shared__ unsigned long long s_dig[16];
    const int kt = blockIdx.x;
    TState &st = g.st[g.sa_btab[kt]];
    const int32_t b0 = g.sa_bstart[kt], b1 = g.sa_bstart[kt + 1];
    long long v[7] = {0, 0, 0, 0, 0, 0, 0};
    unsigned long long dg = 0;  // digests add modulo 2^64
    for (int32_t b = b0 + (int32_t)(blockIdx.y * blockDim.x + threadIdx.x); b < b1;
         b += (int32_t)(gridDim.y * blockDim.x)) {
#pragma unroll
        for (int k = 0; k < 7; ++k) v[k] += g.sa_part[(int64_t)b * 8 + k];
        dg += (unsigned long long)g.sa_part[(int64_t)b * 8 + 7];
    }
    long long tot[7];
#pragma unroll
    for (int k = 0; k < 7; ++k) (void)block_excl_scan64(v[k], tmp, &tot[k]);
    dg = wave_sum64(dg);
    if ((threadIdx.x & 63) == 0) s_dig[threadIdx.x >> 6] = dg;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long d = 0;
        for (int w = 0; w < (int)(blockDim.x >> 6); ++w) d += s_dig[w];
        if (tot[0]) atomicAdd(&st.evicted, (int32_t)tot[0]);
        if (tot[1]) atomicAdd(&st.adm_miss, (int32_t)tot[1]);
        if (tot[2]) atomicAdd(&st.p_fill, (int32_t)tot[2]);
        if (tot[3]) atomicAdd(&st.p_drop, (int32_t)tot[3]);
        if (tot[4]) atomicAdd(&st.m_drop, (int32_t)tot[4]);
        if (tot[5]) atomicAdd(&st.n_res, (int32_t)tot[5]);
        if (tot[6]) atomicAdd(&st.p_res, (int32_t)tot[6]);
        if (d) atomicAdd(&st.digest_acc, d);
    }
}

static inline unsigned grid_for(int64_t n, int per_block, unsigned cap) {
    int64_t b = (n + per_block - 1) / per_block;
    if (b < 1) b = 1;
    if (b > (int64_t)cap) b = cap;
    return (unsigned)b;
}

void launch_sa_place(const DGlobal &g, const PlcParams &p, int64_t nu, int64_t np, int32_t nsa, int64_t blocks1,
                     int64_t blocks, int64_t max_blocks, hipStream_t s) {
    if (nu + np > 0) k_sa_heads<<<grid_for(nu + np, kBlock, 8192), kBlock, 0, s>>>(g, nu, np, p.have_fwd, p.last_stamp);
    // tables of one set per wave come first (fewest sets), then those of two
    if (blocks1 > 0) k_sa_place<1><<<(unsigned)blocks1, kSaBlock, 0, s>>>(g, p, nsa, 0);
    if (blocks > blocks1) k_sa_place<2><<<(unsigned)(blocks - blocks1), kSaBlock, 0, s>>>(g, p, nsa, (int32_t)blocks1);
    // slices: about 4,096 records each for the table with the most blocks
    const unsigned slices = (unsigned)std::min<int64_t>(32, std::max<int64_t>(1, (max_blocks + 4095) / 4096));
    k_sa_sum<<<dim3(nsa, slices), 1024, 0, s>>>(g, nsa);
}

}  // namespace recmg
