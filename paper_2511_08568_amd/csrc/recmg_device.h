// Device-side data layout and helpers of the tiered pooled-embedding lookup.
// Internal to the HIP sources of this package; the public boundary is
// include/recmg.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/recmg.h"

namespace recmg {

constexpr int kBlock = 256;                         // threads per block (4 waves)
constexpr int kWordsPerThread = 4;                  // presence-bitmap words per thread
constexpr int kWordsPerBlock = kBlock * kWordsPerThread;  // 1024 words = 32768 rows
// Tables whose bitmap spans at most kOwnMaxSlices slices of kOwnSliceWords words
// are marked slice by slice in LDS (one block per slice reads the table's ids);
// larger ones with a device atomic per distinct id and block.
constexpr int kOwnSliceWords = 32768;  // 128 KiB of LDS, 2^20 rows
constexpr int kOwnSliceBlocks = kOwnSliceWords / kWordsPerBlock;
#ifndef RECMG_OWN_MAX_SLICES
#define RECMG_OWN_MAX_SLICES 32
#endif
constexpr int kOwnMaxSlices = RECMG_OWN_MAX_SLICES;
__host__ __device__ constexpr bool owns_bitmap(int32_t bm_nblk) { return bm_nblk <= kOwnMaxSlices * kOwnSliceBlocks; }
constexpr int kRadixBits = 11;                      // radix-select digit
constexpr int kRadix = 1 << kRadixBits;
constexpr int32_t kEmpty = -1;                      // map key of a never-used entry
constexpr int32_t kTomb = -2;                       // map key of a deleted entry
constexpr int32_t kPending = INT32_MIN;             // probe result before miss numbering

// per-slot flag bits
constexpr uint32_t F_PF = 1u;    // admitted by a prefetch and not accessed since
constexpr uint32_t F_INP = 4u;   // named by the current placement's prefetch list

// device error flag bits
constexpr int32_t ERR_RANGE = 1;
constexpr int32_t ERR_OFFSETS = 2;
#ifndef RECMG_WPOOL_BAGS
#define RECMG_WPOOL_BAGS 1
#endif
constexpr int kWaveBags = RECMG_WPOOL_BAGS;  // consecutive bags per wave in the wave-per-bag pooled kernel
constexpr int kRaddrPad = 64;  // entries past the batch in the per-index row-address array (read, never used)
constexpr int32_t ERR_INTERNAL = 4;  // a slot-accounting invariant failed (never expected)
// int64 counters of recmg_table_stats_t: kFwdStats of a forward, then the placement's
constexpr int kFwdStats = 7, kPlcStats = 9, kNumStats = kFwdStats + kPlcStats;

// Resident rings: chunks of the buffer whose live entries are counted, and
// the references a zone entry holds besides a slot id.
constexpr int kRingChunk = 1024;
constexpr int32_t kRingHole = INT32_MIN;
constexpr int32_t kRingNewBase = -(1 << 30) - 1;
__host__ __device__ constexpr int32_t ring_ref_miss(int32_t m) { return -1 - m; }            // m < 2^30
__host__ __device__ constexpr int32_t ring_ref_new(int32_t k) { return kRingNewBase - k; }  // k < 2^30 - 1

// outcome of the top-Cap ranking of one table
constexpr int32_t SEL_SELECT = 0;  // keep keys >= threshold
constexpr int32_t SEL_ALL = 1;     // |K| <= Cap: keep everything
constexpr int32_t SEL_NONE = 2;    // Cap == 0 or K empty: keep nothing

// Static description of one table, resident in the workspace.
struct DTable {
    const char *host;      // device-visible pointer to the pinned host table
    char *pool;            // HBM slot pool [cap][row_bytes]
    int32_t *slot_row;     // [cap] row held by the slot, -1 if free
    int32_t *slot_score;   // [cap] ranking score
    uint32_t *slot_flags;  // [cap] F_* bits
    int32_t *slot_touch;   // [cap] stamp of the last forward that hit the slot
    uint8_t *slot_cbit;    // [cap] OR of the caching bits of the last batch (zero between placements)
    int32_t *free_stack;   // [cap] free slot ids, top at free_top
    int2 *map;             // [map_mask + 1] open-addressed row -> slot map (key, slot)
    uint32_t *bitmap;      // [bm_words] presence bitmap, zero between uses
    uint4 *rank;           // [bm_words] (rank of the word's first set bit, word, forward stamp, 0)
                           // written for the non-zero words of a forward's dedup
    int64_t rows;
    int64_t out_elem_off;  // sum of dims of the earlier tables
    int64_t cap_off;       // sum of caps of the earlier tables
    int32_t dim, dtype, row_bytes, cap;
    int32_t map_mask, bm_words, bm_block0, bm_nblk;
    int32_t gsz;           // lanes per bag in the pooled kernel (power of two, 4..64)
    int32_t nchunk;        // element chunks per row in the pooled kernel
    int32_t vec;           // 1: 16-byte vector path, 0: scalar path
    int32_t bags_per_block;
    int32_t copy_unit;     // 16, 4 or 2 bytes
    // wave-per-bag pooled kernel (0 in wlw: not used for this table): each
    // load instruction reads wr rows of 64 / wr lanes x wlw bytes; a row is
    // wnch such chunks
    int32_t wlw, wr, wnch;
    // set-associative form (ways > 0): nsets sets of `ways` slots, row r in set
    // r mod nsets at slots [set * ways, + ways).  Dedup bitmaps index row r at
    // position (set << qbits) | (r / nsets), so sorted distinct rows come out
    // grouped by set, ascending within a set.  ways == 0: fully associative
    // (the map above), bitmap position = row.
    int32_t ways, nsets, qbits;
    int32_t staged;  // 1: misses and prefetch fills of this table are gathered on the host (STAGED)
    int4 *seg;  // [nsets] (U begin, U end, PU begin, PU end) of each set in the
                // current placement, relative to the table's lists; zero between uses
    int32_t *freq;  // LFU_BATCH: [rows] batches that accessed each row (every row, cached or not)
    // LRU_BATCH, fully associative, Cap > 0 (ring_cap > 0): the residents in
    // ascending key order, so that a placement evicts from the front instead
    // of ranking every slot (ring.hip)
    int32_t *slot_pos;  // [cap] index of the slot's entry in the current ring buffer, -1 if none
    int32_t *ring[2];   // [ring_cap] each: slot ids in key order, kRingHole where none; one buffer is
                        // current, the other receives the compacted entries
    int32_t *rcnt[2];   // [ring_cap / kRingChunk] each: live entries per chunk of each buffer
    int32_t *roff;      // [ring_cap / kRingChunk] compaction: first new index of each chunk's entries
    int32_t ring_cap;   // entries per buffer (a multiple of kRingChunk); 0: ranked by radix select
};

// Mutable per-table state and counters, resident in the workspace.
struct TState {
    int32_t ucount;   // distinct rows of the last forward (sorted in U)
    int32_t mcount;   // misses of the last forward (in M, staged at the same index)
    int32_t pcount;   // distinct prefetch rows of the current placement
    int32_t npcount;  // prefetch rows neither resident nor missed (in NP)
    int32_t n_res, free_top, popped, tomb;
    int32_t rebuild, sel_mode, need, plc_nm;  // plc_nm: misses the current placement ranks
    uint64_t prefix;  // radix-select prefix; the threshold key after the last pass
    uint32_t pad0;
    int32_t covered;  // accumulator: distinct prefetch rows of the last placement found in this batch
    // accumulators of the call in flight
    int32_t hits, hits_pf, p_res, evicted, adm_miss, p_fill, p_drop, m_drop;
    unsigned long long digest_acc;
    // resident ring (ring_cap > 0): live entries lie in [r_tail, r_head) of
    // buffer r_buf; r_valid of them are live; this placement evicts the live
    // ones in [r_tail, r_cut).  The rows the last placement's prefetch named
    // (score = this placement's LRU touch) wait in the pending list, entries
    // [pend_off, + pend_n) of pend_row / pend_slot[pend_buf], until a placement
    // merges them into the ring with the rows the last batch touched.
    int32_t r_head, r_tail, r_cut, r_valid, r_buf, r_compact, r_zevict, r_moved;
    int32_t z1_len, z1_keys, pend_n, pend_buf, pend_keep;
    int64_t pend_off;
    // published counters, in recmg_table_stats_t order
    int64_t last[kNumStats];
    unsigned long long digest;
    int64_t total[kNumStats];
};

// Device pointers into the workspace, passed by value to every kernel.
struct DGlobal {
    DTable *tabs;
    TState *st;
    int32_t *err;
    int32_t *bm_block_start;  // [T+1] first bitmap block of each table
    int32_t *blocksum;        // [total bitmap blocks]
    int32_t *blockoff;        // [total bitmap blocks]
    int64_t *tstart;          // [T+1] first index of each table in the last forward
    int64_t *pstart;          // [T+1] first prefetch id of each table in this placement
    int32_t *src;             // [max_indices] per access: slot (>= 0) or -(miss + 1)
    uint64_t *raddr;          // [max_indices] per access: device address of its row (slot or staging)
    int32_t *U;               // [max_indices] sorted distinct rows, table t at tstart[t]
    int32_t *slotU;           // [max_indices] per distinct row: slot or -(miss + 1)
    int32_t *M;               // [max_indices] missed rows, table t at tstart[t]
    uint32_t *mflags;         // [max_indices] F_INP of each miss
    uint8_t *mcbit;           // [max_indices] OR of each miss's caching bits
    int32_t *mscore;          // [max_indices] ranking score of each miss
    int32_t *NP;              // [max_prefetch] new prefetch candidates, table t at pstart[t]
    int32_t *PU;              // [max_prefetch] sorted distinct prefetch rows, table t at pstart[t]
    int32_t *fill_src;        // [max_indices + max_prefetch] admitted row's source: staging row (>= 0)
                              // or -(host row + 1); table t at ftstart[t] + pstart[t]
    int32_t *fill_slot;       // [max_indices + max_prefetch] its slot
    int32_t *hist;            // [T][kRadix]
    int32_t *dump;            // [sum cap] sorted resident rows
    int32_t *dump_count;      // [T]
    char *staging;            // [max_indices][stage_stride] miss rows of the latest forward
                              // (two buffers alternate between forwards; the host picks one)
    int64_t *ftstart;         // [T+1] base of each table's fill list and admitted misses in the
                              // current placement: tstart of the last forward, or 0 if none ran
    int64_t fill_cap;         // entries of fill_src / fill_slot (max_indices + max_prefetch)
    char *fstage;             // [max_prefetch][stage_stride] prefetch rows staged by the host (STAGED)
    int32_t staged_fill;      // 1: some table is STAGED; there a fill source -(k + 1) is fstage row k,
                              // not host row k
    int64_t stage_stride;
    int32_t T;
    int32_t total_bm_blocks;
    int32_t own_tables;  // tables with owns_bitmap(bm_nblk)
    int32_t own_slices;  // the most LDS slices of such a table
    int32_t *sa_bstart;  // [nsa + 1] first placement block of each set-associative table
    int32_t *sa_btab;    // [nsa] those tables, fewest sets first
    int64_t *sa_part;    // [sa blocks][8] each set-associative placement block's counts (added up per table after)
    int32_t *pfrom;      // [max_prefetch] set-associative tables: per distinct prefetch row (PU), its
                         // staging row if the last batch missed it, else -1
    int64_t *stat_log;   // [log calls][T][kNumStats + 1]: the counters of each call (see recmg_stats_log)
    // resident rings (ring.hip)
    int32_t *puref;         // [max_prefetch] per distinct prefetch row (PU) of a fully associative
                            // table: its slot, or ring_ref_miss(m), or ring_ref_new(NP index)
    int2 *zone;             // [max_indices + max_prefetch] (ref, row) of the rows that take the LRU
                            // touch score, in row order; table t at pend_off + tstart[t]
    int32_t *mslot;         // [max_indices] slot admitted for miss m (table t at tstart[t])
    int32_t *npslot;        // [max_prefetch] slot admitted for new candidate k (table t at pstart[t])
    int32_t *pend_row[2];   // [max_prefetch] pending lists (see TState), written by alternate placements
    int32_t *pend_slot[2];  // [max_prefetch] their slots, -1 where the row was not kept
};

// Parameters of one placement.
struct PlcParams {
    int32_t prio;        // 1: PRIORITY
    int32_t es;          // eviction_speed
    int32_t lru_touch;   // LRU score of a row touched by the last batch
    int32_t pscore;      // score of a prefetched row (LFU: 0, a floor that changes nothing)
    int32_t last_stamp;  // stamp of the last forward, -2 if none since the last placement
    int32_t have_fwd;
    int32_t rowbits, total_bits, passes;
    int32_t lfu;         // 1: LFU_BATCH (scores are the rows' batch counts)
};

// Score of a row the last batch touched: LRU_BATCH the batch stamp, PRIORITY
// its caching bit + eviction_speed (Alg. 1), LFU_BATCH its batch count.
__device__ __forceinline__ int32_t touch_score(const PlcParams &p, const DTable &tb, int32_t row, int cbit) {
    if (p.prio) return cbit + p.es;
    if (p.lfu) return tb.freq[row];
    return p.lru_touch;
}

// Score a prefetch gives a row neither resident nor missed.
__device__ __forceinline__ int32_t new_prefetch_score(const PlcParams &p, const DTable &tb, int32_t row) {
    return p.lfu ? tb.freq[row] : p.pscore;
}

// -------------------------------------------------------------------- helpers

// Loads through the global address space.  Pointers read from the workspace
// are generic, and generic (flat) loads also count against the LDS counter, so
// a wave that shuffles between loads would wait for every load in flight.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
#define RECMG_GLOBAL(T, p) (*(const __attribute__((address_space(1))) T *)(p))

__device__ __forceinline__ uint4 gload16(const void *p) {
    const u32x4_t v = RECMG_GLOBAL(u32x4_t, p);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ uint32_t gload4(const void *p) { return RECMG_GLOBAL(uint32_t, p); }
__device__ __forceinline__ uint16_t gload2(const void *p) { return RECMG_GLOBAL(uint16_t, p); }
__device__ __forceinline__ int2 gload_int2(const void *p) {
    const i32x2_t v = RECMG_GLOBAL(i32x2_t, p);
    return make_int2(v[0], v[1]);
}

__device__ __forceinline__ uint32_t hash_row(int32_t r) {
    // murmur3 32-bit finaliser
    uint32_t h = (uint32_t)r;
    h ^= h >> 16;
    h *= 0x85ebca6bu;
    h ^= h >> 13;
    h *= 0xc2b2ae35u;
    h ^= h >> 16;
    return h;
}

// Slot of `row` or -1.  Linear probing; deleted entries are skipped.
__device__ __forceinline__ int32_t map_find(const DTable &tb, int32_t row) {
    const int32_t mask = tb.map_mask;
    uint32_t i = hash_row(row) & (uint32_t)mask;
    for (int32_t n = 0; n <= mask; ++n) {
        const int2 e = gload_int2(tb.map + i);
        if (e.x == row) return e.y;
        if (e.x == kEmpty) return -1;
        i = (i + 1) & (uint32_t)mask;
    }
    return -1;
}

// The map holds at most Cap live rows in >= 4 Cap entries, and is rebuilt when
// deleted entries pass a quarter of it, so at least half of it stays empty.

// Insert a row known to be absent.  Concurrent inserts of distinct rows are
// safe; no lookup may run concurrently.  Returns 1 if a deleted entry was reused.
__device__ __forceinline__ int map_insert(const DTable &tb, int32_t row, int32_t slot) {
    const int32_t mask = tb.map_mask;
    uint32_t i = hash_row(row) & (uint32_t)mask;
    for (int32_t n = 0; n <= mask; ++n) {
        int32_t k = tb.map[i].x;  // may be stale (L1); the CAS result is not
        while (k == kEmpty || k == kTomb) {
            const int32_t prev = atomicCAS(&tb.map[i].x, k, row);
            if (prev == k) {
                tb.map[i].y = slot;
                return k == kTomb;
            }
            k = prev;  // lost the entry to another insert
        }
        i = (i + 1) & (uint32_t)mask;
    }
    return 0;
}

// Delete a present row (distinct rows may be deleted concurrently).
__device__ __forceinline__ void map_delete(const DTable &tb, int32_t row) {
    const int32_t mask = tb.map_mask;
    uint32_t i = hash_row(row) & (uint32_t)mask;
    for (int32_t n = 0; n <= mask; ++n) {
        int32_t k = tb.map[i].x;
        if (k == row) {
            tb.map[i].x = kTomb;
            return;
        }
        if (k == kEmpty) return;
        i = (i + 1) & (uint32_t)mask;
    }
}

// Bitmap position of row r (see DTable::qbits) and its inverse.
__device__ __forceinline__ uint32_t bm_pos(int32_t nsets, int32_t qbits, int32_t r) {
    if (!nsets) return (uint32_t)r;
    const uint32_t u = (uint32_t)r, n = (uint32_t)nsets;
    return ((u % n) << qbits) | (u / n);
}
__device__ __forceinline__ uint32_t bm_pos(const DTable &tb, int32_t r) { return bm_pos(tb.nsets, tb.qbits, r); }
__device__ __forceinline__ int32_t bm_row(const DTable &tb, uint32_t pos) {
    if (!tb.nsets) return (int32_t)pos;
    return (int32_t)((pos & ((1u << tb.qbits) - 1u)) * (uint32_t)tb.nsets + (pos >> tb.qbits));
}

// Slot of `row` in its set, or -1.
__device__ __forceinline__ int32_t set_find(const DTable &tb, int32_t row) {
    const int32_t base = (int32_t)((uint32_t)row % (uint32_t)tb.nsets) * tb.ways;
    for (int32_t k = 0; k < tb.ways; ++k)
        if ((int32_t)gload4(tb.slot_row + base + k) == row) return base + k;
    return -1;
}

__device__ __forceinline__ int32_t find_slot(const DTable &tb, int32_t row) {
    return tb.ways ? set_find(tb, row) : map_find(tb, row);
}

// SplitMix64 output mix (Steele, Lea & Flood, OOPSLA 2014).
__device__ __forceinline__ unsigned long long mix64(unsigned long long z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

// Largest t in [0, T) with starts[t] <= i (starts non-decreasing).
__device__ __forceinline__ int find_seg(const int64_t *starts, int T, int64_t i) {
    int lo = 0, hi = T - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (starts[mid] <= i) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int find_seg32(const int32_t *starts, int T, int32_t i) {
    int lo = 0, hi = T - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (starts[mid] <= i) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ int wave_incl_scan(int x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        int y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    return x;
}

// Exclusive scan over the block (blockDim.x a multiple of 64, <= 1024).
// `tmp` is __shared__ int[16]; every thread must call.
__device__ __forceinline__ int block_excl_scan(int v, int *tmp, int *total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int x = wave_incl_scan(v);
    if (lane == 63) tmp[wid] = x;
    __syncthreads();
    int pre = 0, tot = 0;
    for (int k = 0; k < nw; ++k) {
        int s = tmp[k];
        pre += (k < wid) ? s : 0;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return pre + x - v;
}

// 64-bit exclusive scan over the block; `tmp` is __shared__ long long[16].
__device__ __forceinline__ long long block_excl_scan64(long long v, long long *tmp, long long *total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    long long x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const long long y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) tmp[wid] = x;
    __syncthreads();
    long long pre = 0, tot = 0;
    for (int k = 0; k < nw; ++k) {
        const long long s = tmp[k];
        pre += (k < wid) ? s : 0;
        tot += s;
    }
    __syncthreads();
    *total = tot;
    return pre + x - v;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) v += __shfl_xor(v, d, 64);
    return v;
}

__device__ __forceinline__ unsigned long long wave_sum64(unsigned long long v) {
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) {
        unsigned lo = __shfl_xor((unsigned)v, d, 64);
        unsigned hi = __shfl_xor((unsigned)(v >> 32), d, 64);
        v += ((unsigned long long)hi << 32) | lo;
    }
    return v;
}

// Sum over the block; result valid in every thread.  `tmp` is __shared__ int[16].
__device__ __forceinline__ int block_sum(int v, int *tmp) {
    int dummy;
    int excl = block_excl_scan(v, tmp, &dummy);
    (void)excl;
    return dummy;
}

// Append for the lanes with `want`, to the counter of their own table:
// returns each such lane's index (one atomic per table present in the wave).
// Every lane of the wave must call.
__device__ __forceinline__ int32_t wave_append(bool want, int t, int32_t *counter0, int counter_stride) {
    const int lane = threadIdx.x & 63;
    const unsigned long long below = (1ull << lane) - 1ull;
    unsigned long long pending = __ballot(want);
    int32_t mine = -1;
    while (pending) {
        const int leader = __ffsll((long long)pending) - 1;
        const int lt = __shfl(t, leader, 64);
        const unsigned long long grp = __ballot(want && t == lt);
        int32_t base = 0;
        if (lane == leader) base = atomicAdd(counter0 + (int64_t)lt * counter_stride, (int32_t)__popcll(grp));
        base = __shfl(base, leader, 64);
        if (want && t == lt) mine = base + (int32_t)__popcll(grp & below);
        pending &= ~grp;
    }
    return mine;
}

// This block's contiguous share [*lo, *hi) of an index space of n, in whole
// blocks of blockDim.x: a block then meets one or two tables, and its LDS
// counters reach the table states with one or two atomics.
__device__ __forceinline__ void block_share(int64_t n, int64_t *lo, int64_t *hi) {
    const int64_t per = ((n + gridDim.x - 1) / gridDim.x + blockDim.x - 1) / blockDim.x * blockDim.x;
    *lo = (int64_t)blockIdx.x * per;
    *hi = *lo + per < n ? *lo + per : n;
}

// Count the lanes with `want` into their own table's LDS counter, one LDS
// atomic per table present in the wave.  Counts that only add up go through
// LDS and reach the table's state once per block: a global atomic from every
// wave would queue on the few lines of the table's state.  Every lane of the
// wave must call.
__device__ __forceinline__ void wave_count_lds(bool want, int t, int *s_cnt) {
    const int lane = threadIdx.x & 63;
    unsigned long long pending = __ballot(want);
    while (pending) {
        const int leader = __ffsll((long long)pending) - 1;
        const int lt = __shfl(t, leader, 64);
        const unsigned long long grp = __ballot(want && t == lt);
        if (lane == leader) atomicAdd(&s_cnt[lt], (int)__popcll(grp));
        pending &= ~grp;
    }
}

__device__ __forceinline__ uint64_t make_key(int32_t score, int32_t row, int rowbits) {
    return ((uint64_t)(uint32_t)score << rowbits) | (uint64_t)(uint32_t)row;
}

// The error word read once per block.  Evict and admit may set it (a broken
// invariant) while other blocks of the same kernel start, and the waves of a
// block must agree before the block's barriers.
__device__ __forceinline__ bool block_err(const DGlobal &g) {
    __shared__ int s_err;
    if (threadIdx.x == 0) s_err = *g.err;
    __syncthreads();
    return s_err != 0;
}

// A placement's candidate counts for table t: |K| = residents + the last
// batch's misses + new prefetch rows, of which min(Cap, |K|) stay.
struct Counts {
    int32_t cap, nm, nnp, mode, keep;
};

__device__ __forceinline__ Counts table_counts(const DTable &tb, const TState &st, const PlcParams &p) {
    Counts c;
    c.cap = tb.cap;
    c.nm = p.have_fwd ? st.mcount : 0;
    c.nnp = st.npcount;
    const int64_t nk = (int64_t)st.n_res + c.nm + c.nnp;
    c.keep = (int32_t)(nk < c.cap ? nk : c.cap);
    c.mode = nk <= c.cap ? SEL_ALL : (c.keep == 0 ? SEL_NONE : SEL_SELECT);
    return c;
}

__device__ __forceinline__ bool kept(int mode, uint64_t key, uint64_t thr) {
    return mode == SEL_ALL || (mode == SEL_SELECT && key >= thr);
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __builtin_bit_cast(float, bits16 << 16);
}

__device__ __forceinline__ float f16_to_f32(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

// Copy `count[t]` rows of every table in 16/4/2-byte units, the tables' work
// laid end to end so every table gets its share of the first `nblocks` blocks
// of the grid (the others copy nothing).  src_of / dst_of give the byte
// addresses of item j of table t.
template <class Src, class Dst>
__device__ __forceinline__ void copy_flat(const DGlobal &g, const int32_t *count, int64_t nblocks, Src src_of,
                                          Dst dst_of) {
    __shared__ int64_t s_pre[RECMG_MAX_TABLES + 1];
    __shared__ long long tmp[16];
    // per-table unit counts, scanned (T <= 256 = blockDim)
    long long mine = 0;
    const int t0 = threadIdx.x;
    if (t0 < g.T) mine = (long long)count[t0] * (g.tabs[t0].row_bytes / g.tabs[t0].copy_unit);
    long long tot;
    const long long ex = block_excl_scan64(mine, tmp, &tot);
    if (t0 < g.T) s_pre[t0] = ex;
    if (t0 == 0) s_pre[g.T] = tot;
    __syncthreads();
    const int64_t items = (int64_t)blockIdx.x < nblocks ? s_pre[g.T] : 0;
    const int64_t S = nblocks * blockDim.x;
    for (int64_t base = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; base < items; base += 4 * S) {
        uint4 v16[4];
        uint32_t v4[4];
        uint16_t v2[4];
        char *dst[4];
        int unit[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            dst[q] = nullptr;
            unit[q] = 0;
            const int64_t it = base + q * S;
            if (it < items) {
                const int t = find_seg(s_pre, g.T, it);
                const DTable &tb = g.tabs[t];
                const int u = tb.copy_unit, nunit = tb.row_bytes / u;
                const int64_t loc = it - s_pre[t];
                const int64_t j = loc / nunit;
                const int64_t vo = (loc - j * nunit) * u;
                const char *sp = src_of(t, tb, j) + vo;
                dst[q] = dst_of(t, tb, j) + vo;
                unit[q] = u;
                if (u == 16) v16[q] = gload16(sp);
                else if (u == 4) v4[q] = gload4(sp);
                else v2[q] = gload2(sp);
            }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (unit[q] == 16) *reinterpret_cast<uint4 *>(dst[q]) = v16[q];
            else if (unit[q] == 4) *reinterpret_cast<uint32_t *>(dst[q]) = v4[q];
            else if (unit[q] == 2) *reinterpret_cast<uint16_t *>(dst[q]) = v2[q];
        }
    }
}

}  // namespace recmg
