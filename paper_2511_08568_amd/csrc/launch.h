// Host-side launchers of the kernels, one group per translation unit.
#pragma once

#include "recmg_device.h"

namespace recmg {

// Up to this many items, a grid-stride launch gives each thread one item (a
// short batch is latency-bound: its threads' dependent load chains run side
// by side instead of one after another); above, `big` items per thread.
constexpr int64_t kTinyItems = 16384;
static inline int items_per_thread(int64_t n, int big) { return n <= kTinyItems ? 1 : big; }

// dedup.hip
void launch_mark(const DGlobal &g, const int32_t *keys, const int64_t *starts, int64_t n, hipStream_t s);
void launch_mark_resident(const DGlobal &g, int32_t max_cap, hipStream_t s);
enum { EMIT_FORWARD = 0, EMIT_PREFETCH = 1, EMIT_DUMP = 2 };
// mode: where the sorted distinct ids go (U of a forward, PU of a placement, the resident dump);
// max_nblk: the most bitmap blocks of any table (at most kFusedMaxBlocks: one kernel does it all)
constexpr int kFusedMaxBlocks = 8;
void launch_dedup(const DGlobal &g, int mode, int32_t *counts, int count_stride, int32_t stamp, int32_t max_nblk,
                  hipStream_t s);

// forward.hip
void launch_fwd_prep(const DGlobal &g, const int64_t *offsets, int32_t B, int64_t n, hipStream_t s);
void launch_fwd_probe(const DGlobal &g, int32_t stamp, int64_t n, hipStream_t s);
void launch_fwd_src(const DGlobal &g, const int32_t *indices, int64_t n, hipStream_t s);
void launch_fwd_cover(const DGlobal &g, int32_t stamp, int64_t np, hipStream_t s);
// ev0 / ev1 (may be null): recorded by the dispatch itself around the kernel
void launch_fetch(const DGlobal &g, hipStream_t s, hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// Pooled-sum kernels: kinds [0, kPoolKindsGroup) are the group-per-bag kernel
// (dtype * 2 + vec), the rest the wave-per-bag kernel per (dtype, wlw, wr).
constexpr int kPoolKindsGroup = 6, kPoolKinds = kPoolKindsGroup + 15;
int pool_kind(int dtype, int vec, int wlw, int wr);
// one launch per kind present, over the blocks [boff, boff + nblk) of the
// tables btab[k] ordered by kind; bstart[k] = first block of btab[k].  The
// launch's tables are btab[k0 ..]; wave-per-bag kinds give every table the
// same number of blocks, nbt.
struct PoolLaunch {
    int32_t kind, boff, nblk, k0, nbt;
};
void launch_pool(const DGlobal &g, const int64_t *offsets, int32_t B, float *out, const int32_t *bstart,
                 const int32_t *btab, int32_t nt, const PoolLaunch *ls, int nl, hipEvent_t ev0, hipEvent_t ev1,
                 hipStream_t s);
// log_slot: record of this call in the stats log, or -1
void launch_fwd_finalize(const DGlobal &g, int64_t log_slot, hipStream_t s);

// placement.hip
void launch_plc_prep(const DGlobal &g, const int64_t *poff, int64_t np, int32_t have_fwd, hipStream_t s);
void launch_plc_bits(const DGlobal &g, const uint8_t *bits, int64_t n_last, hipStream_t s);
void launch_plc_freq(const DGlobal &g, int64_t n_last, hipStream_t s);
void launch_plc_classify(const DGlobal &g, int32_t last_stamp, int64_t np, hipStream_t s);
// item_bound: the most slots + candidates of any table; up to kRankSmallItems one
// block per table ranks it whole
constexpr int64_t kRankSmallItems = 1 << 16;
void launch_plc_rank(const DGlobal &g, const PlcParams &p, int64_t item_bound, hipStream_t s);
// evict (tables ranked by radix select), then map upkeep and admission (every
// fully associative table)
void launch_plc_evict(const DGlobal &g, const PlcParams &p, int32_t max_cap, hipStream_t s);
void launch_plc_admit(const DGlobal &g, const PlcParams &p, int32_t max_cap, int32_t max_map, int64_t cand_bound,
                      hipStream_t s);
// fdesc: this placement's fill descriptor, [T][4] int64 (written by finalize, read by fill);
// phase: the tables whose rows this launch copies, by miss mode
enum { FILL_ZERO_COPY = 1, FILL_STAGED = 2 };
void launch_plc_fill(const DGlobal &g, const int64_t *fdesc, int phase, hipStream_t s, hipEvent_t ev0 = nullptr,
                     hipEvent_t ev1 = nullptr);
void launch_plc_finalize(const DGlobal &g, int64_t *fdesc, int64_t log_slot, hipStream_t s);
void launch_init_state(const DGlobal &g, int32_t max_cap, hipStream_t s);

// ring.hip: LRU_BATCH placement of tables with a resident ring (ring_cap > 0).
// item_bound: entries of a table's zones and prefetch list (last forward's
// distinct rows + pending rows + prefetch rows, per table); ring_chunks: the
// most kRingChunk chunks of any ring; wr: the pending buffer this placement
// writes (the next one reads it).
void launch_ring_rank(const DGlobal &g, const PlcParams &p, int64_t item_bound, hipStream_t s);
void launch_ring_evict(const DGlobal &g, const PlcParams &p, int64_t item_bound, int32_t ring_chunks, hipStream_t s);
void launch_ring_store(const DGlobal &g, const PlcParams &p, int64_t item_bound, int32_t max_cap, int wr,
                       hipStream_t s);

// setassoc.hip: placement of the set-associative tables (nu: index space of
// the last forward's distinct rows, np: of this placement's prefetch rows;
// nsa tables, fewest sets first; blocks = sa_bstart[nsa], the first blocks1 of
// them over tables of one set per wave), kSaWaves * sa_sets_per_wave(ways,
// nsets) sets per block of a table
constexpr int kSaWaves = 16, kSaBlock = 64 * kSaWaves;
// sets per wave of a table: two (32 lanes each) when the ways fit in half a
// wave and the sets are many (few events each); one where sets take many events
constexpr int64_t kSaPairMinSets = 16384;
constexpr int sa_sets_per_wave(int ways, int64_t nsets) { return ways <= 32 && nsets >= kSaPairMinSets ? 2 : 1; }
// max_blocks: the most blocks of one table (sizes the per-table sum of the blocks' counts)
void launch_sa_place(const DGlobal &g, const PlcParams &p, int64_t nu, int64_t np, int32_t nsa, int64_t blocks1,
                     int64_t blocks, int64_t max_blocks, hipStream_t s);

}  // namespace recmg
