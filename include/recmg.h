/*
 * recmg.h -- C ABI of the tiered pooled-embedding lookup for MI355X (gfx950).
 *
 * The operation is the one RecMG's caching and prefetching decisions act on
 * (arXiv 2511.08568): a per-batch pooled embedding-bag lookup (Sec. II: the
 * rows a feature touches are gathered from an embedding table and combined by
 * summation) over a two-tier store.  Every table lives whole in pinned host
 * DRAM; a software-managed cache of rows lives in HBM (Sec. I, Sec. VI-B).
 * Residency is decided between batches from two caller-supplied inputs, the
 * per-access caching bits and the prefetch list (Sec. VI-B, VI-C), applied
 * once each batch ends by Alg. 1 (load_embeddings) and Alg. 2
 * (gpu_buffer_populate).
 *
 * Cache semantics, per table t (fully associative, one cache per table;
 * config.ways selects the set-associative form below):
 *   keys are (score, row); the cache keeps the min(Cap_t, |K|) largest keys of
 *   K = resident ∪ last batch's misses ∪ set(prefetch list); among equal
 *   scores the lower row id is evicted first.
 *   LRU_BATCH: a row's score is the batch that last touched it; a prefetch
 *   before batch b scores b.
 *   PRIORITY (Alg. 1 / Alg. 2): residents age by one (saturating at 0) per
 *   placement; a touched row scores bit + eviction_speed, with bit the OR of
 *   its caching bits in the last batch; a prefetched row scores
 *   max(its score, eviction_speed).
 *   LFU_BATCH (the LFU baseline of Sec. VII-B, per batch): a row's score is
 *   the number of batches that have accessed it, counted for every row
 *   whether cached or not (a device array of N_t counters) by the placement
 *   that consumes the batch (a batch no placement follows is not counted);
 *   a prefetch does not change it.
 *
 * Set-associative form (config.ways = W > 0; the production buffer of Sec.
 * VI-B is a W-way set-associative software cache, Sec. VII-B and VII-E): a
 * table has S = floor(Cap_t / W) sets of W slots (Cap_t mod W slots unused; S
 * = 0 caches nothing) and row r belongs to set r mod S.  Alg. 1 and Alg. 2
 * run literally inside each set: rows the last batch touched take the touch
 * score (no aging); then the set's misses, ascending by row, and the set's
 * distinct prefetch rows, ascending, are inserted (a resident prefetched row
 * only keeps max(score, prefetch score)).  An insertion takes the lowest free
 * slot of the set; in a full set, the lowest slot holding the minimum score
 * is the victim and, under PRIORITY, every slot of the set then ages by one
 * (saturating at 0).  A row that ends in a slot other than the one it started
 * in has prefetch flag [row in P]; such a row, when it was resident before and
 * moved, is read from the host again and counts in prefetch_fill.
 *
 * Call order:  recmg_cache_init -> { recmg_apply_placement ->
 *              recmg_embbag_forward }* -> recmg_stats -> recmg_cache_destroy.
 * A placement consumes the distinct rows and misses of the most recent
 * forward (none if no forward ran since the previous placement).
 *
 * Threading and streams: one handle must not be used from two host threads at
 * once.  All device work of a call is enqueued on the `stream` argument (a
 * hipStream_t, NULL = the null stream); only recmg_stats and the STAGED miss
 * path synchronise with the host.
 *
 * Errors: every entry point returns a recmg_status_t.  Argument errors found
 * on the host leave the cache state unchanged.  An error returned after a
 * placement or forward has begun enqueuing device work (RECMG_E_HIP, or
 * RECMG_E_STATE from the STAGED host path) leaves the device state ahead of
 * the handle's own bookkeeping: the handle is then broken, every later call
 * but recmg_cache_destroy returns RECMG_E_STATE, and it must be destroyed.
 * Out-of-range rows found on the device (validate = 0) latch a device error
 * flag: that call and every later call become no-ops on the device, and the
 * next recmg_stats returns RECMG_E_RANGE.  With validate = 1 the host copies the ids back and checks
 * them before anything is launched (synchronous; for debugging).
 * recmg_last_error() gives a message for the calling thread's last error.
 */
#ifndef RECMG_H
#define RECMG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RECMG_MAX_TABLES 256

typedef enum {
    RECMG_OK = 0,
    RECMG_E_INVALID = 1, /* null, inconsistent or over-size argument */
    RECMG_E_RANGE = 2,   /* a row id outside [0, rows_t) or malformed offsets */
    RECMG_E_STATE = 3,   /* call on a destroyed or broken handle, or a broken invariant */
    RECMG_E_HIP = 4,     /* HIP runtime error (message via recmg_last_error) */
    RECMG_E_NOMEM = 5    /* workspace or staging buffer smaller than queried */
} recmg_status_t;

typedef enum { RECMG_F32 = 0, RECMG_F16 = 1, RECMG_BF16 = 2 } recmg_dtype_t;
typedef enum { RECMG_LRU_BATCH = 0, RECMG_PRIORITY = 1, RECMG_LFU_BATCH = 2 } recmg_policy_t;
typedef enum {
    RECMG_ZERO_COPY = 0, /* misses are read from host memory by a GPU kernel over the host link */
    RECMG_STAGED = 1     /* miss ids (and the placement's prefetch fills) go to the host, a
                            host gather packs rows into pinned staging, and one copy per table
                            moves them on the copy stream; the GPU never reads host tables */
} recmg_miss_mode_t;

typedef struct recmg_cache recmg_cache_t; /* opaque handle */

/* Configuration.  All arrays are host memory of length num_tables and are
 * only read during recmg_query_workspace / recmg_cache_init. */
typedef struct {
    int32_t num_tables;                 /* 1 .. RECMG_MAX_TABLES */
    const int64_t *rows;                /* N_t, 1 .. 2^31-1 */
    const int32_t *dims;                /* D_t >= 1 (elements per row) */
    const int32_t *dtypes;              /* recmg_dtype_t per table */
    const void *const *host_tables;     /* row-major [N_t][D_t], caller-owned, read-only while
                                           the handle lives.  ZERO_COPY: pinned host memory
                                           (hipHostMalloc / torch pin_memory), 16-byte aligned
                                           when D_t*elem is a multiple of 16; the GPU reads it.
                                           STAGED: any host memory; only the host reads it */
    const int64_t *cache_rows;          /* Cap_t >= 0 HBM slots (clamped to N_t) */
    int32_t policy;                     /* recmg_policy_t */
    int32_t eviction_speed;             /* PRIORITY only; 0 .. 1<<20 (the paper uses 4) */
    int32_t miss_mode;                  /* recmg_miss_mode_t */
    int32_t validate;                   /* 1: synchronous host-side range checks */
    int32_t max_bags_per_table;         /* upper bound on bags_per_table of any forward */
    int64_t max_indices;                /* upper bound on num_indices of any forward */
    int64_t max_prefetch;               /* upper bound on num_prefetch of any placement */
    void *device_workspace;             /* caller-owned device memory (e.g. a torch uint8
                                           tensor), >= the queried size, 256-byte aligned */
    size_t device_workspace_bytes;
    void *host_staging;                 /* caller-owned pinned host memory, STAGED only */
    size_t host_staging_bytes;
    void *copy_stream;                  /* hipStream_t for STAGED copies and the placement's
                                           fill; NULL = the stream of each call */
    int32_t timing;                     /* initial timing level (see recmg_set_timing): 0 none,
                                           1 the pooled, fetch and fill kernels, 2 every stage */
    int32_t ways;                       /* 0: fully associative caches.  1 .. 64: W-way
                                           set-associative caches (see below) */
    int32_t stats_log_calls;            /* >= 0: the counters of the latest this many calls
                                           are kept on the device (recmg_stats_log) */
    const int32_t *miss_modes;          /* NULL: every table in miss_mode.  Else per table
                                           (recmg_miss_mode_t): ZERO_COPY tables must be pinned
                                           and are read by the GPU, STAGED tables are gathered on
                                           the host (e.g. pin the tables the host allows and
                                           leave the rest pageable); the two run side by side */
} recmg_config_t;

/* Stages timed at timing level 2 (at level 1: the kernels named in
 * recmg_set_timing). */
typedef enum {
    RECMG_STAGE_FWD_DEDUP = 0,  /* offsets check, dedup + sort, map probe, inverse map */
    RECMG_STAGE_FWD_FETCH = 1,  /* on-demand miss fetch (zero-copy kernel or staged copy) */
    RECMG_STAGE_FWD_POOL = 2,   /* pooled gather + sum */
    RECMG_STAGE_PLC_CLASSIFY = 3, /* caching bits, prefetch dedup + classification */
    RECMG_STAGE_PLC_RANK = 4,   /* scoring + radix select of the kept keys (LRU_BATCH fully
                                   associative tables: new scores, zones and the cut of the
                                   resident ring) */
    RECMG_STAGE_PLC_APPLY = 5,  /* evict, map maintenance, admit, counters */
    RECMG_STAGE_PLC_FILL = 6,   /* copy of admitted rows into slots (host link for prefetch) */
    RECMG_STAGE_HOST_LINK = 7,  /* union of the FWD_FETCH and PLC_FILL intervals: the time the host
                                   link was in use (the two can overlap on different streams) */
    RECMG_NUM_STAGES = 8
} recmg_stage_t;

/* Counters of one table.  The first group describes a forward, the second a
 * placement (Sec. VII-E splits accesses into hits from caching, hits from
 * prefetching and on-demand fetches).  Prefetch quality (Sec. IV, Eq. coverage;
 * Sec. VII-E): coverage = prefetch_covered / unique of a forward, with P the
 * prefetch list of the placement just before it; prefetch accuracy (the
 * prefetched rows the next batch uses, over the rows prefetched) =
 * prefetch_covered / prefetch_distinct, summed over placement + forward pairs.
 * Both depend only on the lists and the batches, not on the cache. */
typedef struct {
    int64_t lookups;           /* indices of this table in the batch */
    int64_t unique;            /* distinct rows U */
    int64_t hits;              /* |U ∩ R| */
    int64_t hits_prefetch;     /* hits on rows still flagged as prefetched: admitted while the
                                  prefetch list named them (from the host, or from staging as a
                                  miss of the batch before) and not accessed since */
    int64_t misses;            /* |U \ R| = on-demand fetches, each row fetched once */
    int64_t ondemand_bytes;    /* misses * row bytes */
    int64_t prefetch_covered;  /* |set(P) ∩ U|, P of the placement just before this forward
                                  (0 if another forward came between) */
    int64_t evicted;           /* |R \ R'| */
    int64_t admitted_miss;     /* |(R' \ R) ∩ M| */
    int64_t prefetch_fill;     /* |(R' \ R) \ M|: rows fetched from host for prefetch */
    int64_t prefetch_resident; /* |P ∩ R| */
    int64_t prefetch_dropped;  /* |P \ (R ∪ R')| */
    int64_t miss_dropped;      /* |M \ R'| */
    int64_t resident;          /* |R'| */
    int64_t prefetch_bytes;    /* prefetch_fill * row bytes */
    int64_t prefetch_distinct; /* |set(P)| */
    uint64_t digest;           /* sum over R' of SplitMix64-mix((t << 40) | row) mod 2^64 */
} recmg_table_stats_t;

/* Sizes the caller must provide: device workspace bytes and, for STAGED,
 * pinned host staging bytes (0 for ZERO_COPY).  Pure function of *cfg (the
 * workspace/staging pointers and sizes in *cfg are ignored). */
int32_t recmg_query_workspace(const recmg_config_t *cfg, size_t *device_bytes, size_t *host_staging_bytes);

/* Creates a handle on the current HIP device: checks the configuration, maps
 * the host tables for device access, carves the workspace and clears it
 * (synchronously).  The cache starts empty.  *out is set only on success. */
int32_t recmg_cache_init(const recmg_config_t *cfg, recmg_cache_t **out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): as
 * recmg_cache_init, but the workspace is a fixed 32 MiB array inside the
 * library, one per device (held from the library's first use of it on that
 * device until the process ends); cfg->device_workspace and
 * device_workspace_bytes are ignored.  Nothing is allocated on the device.
 * The host staging buffer (STAGED) still comes from the caller.
 *   RECMG_E_NOMEM   the configuration's workspace (recmg_query_workspace) is
 *                   larger than 32 MiB;
 *   RECMG_E_STATE   another live handle of this device holds the array (at
 *                   most one at a time; recmg_cache_destroy releases it).
 * The array keeps what the last handle left in it; init clears everything a
 * handle reads before writing it.  All calls on the handle use the array, so
 * calls that overlap on one device race only as calls on one handle would
 * (they are ordered by the handle's events). */
int32_t recmg_cache_init_static(const recmg_config_t *cfg, recmg_cache_t **out);

/* Placement before the next forward (Alg. 1 + Alg. 2, batched: one ranking
 * per placement).
 *   prefetch_rows     device int32 [num_prefetch], table-major, may repeat ids;
 *   prefetch_offsets  device int64 [num_tables + 1], prefetch_offsets[0] = 0,
 *                     prefetch_offsets[T] = num_prefetch;
 *   num_prefetch      host count, 0 .. max_prefetch;
 *   cache_bits        device uint8, one per index of the most recent forward
 *                     (non-zero = 1), or NULL (all 0).  Ignored by LRU_BATCH.
 * Arrays may be freed or reused once the stream has passed this call. */
int32_t recmg_apply_placement(recmg_cache_t *c, const int32_t *prefetch_rows, const int64_t *prefetch_offsets,
                              int64_t num_prefetch, const uint8_t *cache_bits, void *stream);

/* Pooled lookup of one batch (Sec. II, summation).
 *   indices         device int32 [num_indices], table-major;
 *   offsets         device int64 [num_tables * bags_per_table + 1], bag j of
 *                   table t is indices[offsets[t*B + j] .. offsets[t*B + j + 1]);
 *                   offsets[0] = 0, non-decreasing, last = num_indices;
 *   out             device float32, table-major [T][B][D_t]; written whole
 *                   (an empty bag gives zeros).  Sums accumulate in fp32 in a
 *                   fixed order per bag, so results do not depend on which
 *                   tier served a row.
 * Misses are fetched once per distinct row (ZERO_COPY: GPU reads of pinned
 * host memory; STAGED: host gather + copy on the copy stream, synchronising
 * the host once). */
int32_t recmg_embbag_forward(recmg_cache_t *c, const int32_t *indices, const int64_t *offsets,
                             int64_t num_indices, int32_t bags_per_table, float *out, void *stream);

/* Synchronises the last stream used, then copies counters to host memory:
 *   last   [num_tables] counters of the most recent forward / placement, or NULL;
 *   total  [num_tables] sums over all calls (digest = the latest), or NULL;
 *   resident_dump    host int32 [dump_capacity] or NULL: resident rows of every
 *                    table, table after table, ascending within a table;
 *   resident_counts  host int64 [num_tables] or NULL: rows per table in the dump.
 * Returns RECMG_E_INVALID (nothing written to the dump) if dump_capacity is
 * too small, RECMG_E_RANGE if the device error flag is set. */
int32_t recmg_stats(recmg_cache_t *c, recmg_table_stats_t *last, recmg_table_stats_t *total,
                    int32_t *resident_dump, int64_t dump_capacity, int64_t *resident_counts);

/* Counters of individual calls, in call order (placements and forwards
 * numbered together from 0), from the device log of the latest
 * config.stats_log_calls calls (the per-batch log a6 of the stats row: Sec.
 * VII-E's access split per batch).  Synchronises.
 *   out         host [n_calls][num_tables]: record of call first_call + k, table t
 *               at out[k * num_tables + t].  A placement's record holds its
 *               placement counters and the digest after it, a forward's record
 *               its forward counters; the other group and a forward's digest are 0.
 *   calls_made  host, or NULL: number of calls so far.
 * RECMG_E_INVALID if a requested call is not (or no longer) in the log;
 * n_calls = 0 only reports calls_made. */
int32_t recmg_stats_log(recmg_cache_t *c, recmg_table_stats_t *out, int64_t first_call, int64_t n_calls,
                        int64_t *calls_made);

/* Device time per stage, summed over the calls since the last reset, in
 * milliseconds (ms[RECMG_NUM_STAGES]), and how many times each stage ran
 * (calls[RECMG_NUM_STAGES], may be NULL).  Synchronises.  reset != 0 clears
 * the sums afterwards.  Only stages timed at the level in force when a call
 * ran are counted (see recmg_set_timing). */
int32_t recmg_stage_times(recmg_cache_t *c, double *ms, int64_t *calls, int32_t reset);

/* Timing level for later calls:
 *   0  none;
 *   1  the kernels of the pooled sum, of the zero-copy miss fetch and of the
 *      placement's fill (RECMG_STAGE_FWD_POOL, _FWD_FETCH, _PLC_FILL, and
 *      their host-link union), by events their own dispatches record (no
 *      command is added to the stream; such a dispatch starts a little later,
 *      by a few microseconds);
 *   2  every stage: an event pair per stage per call around the stage's
 *      commands (two extra stream commands per stage, a few microseconds each).
 * Returns RECMG_E_INVALID for another level.  Not thread-safe with calls in
 * flight on another host thread (the handle is single-threaded anyway). */
int32_t recmg_set_timing(recmg_cache_t *c, int32_t level);

/* Waits for outstanding work and releases the handle (not the caller's
 * buffers).  NULL is accepted. */
int32_t recmg_cache_destroy(recmg_cache_t *c);

/* Message of the calling thread's last error ("" if none). */
const char *recmg_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RECMG_H */
