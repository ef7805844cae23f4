// C ABI of include/recmg.h: configuration checks, workspace carving, launch
// order, the STAGED miss path and counter readback.  All arithmetic of the
// lookup runs in the kernels of dedup.hip, forward.hip and placement.hip.
#include <algorithm>
#include <atomic>
#include <cstddef>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "launch.h"

using namespace recmg;

namespace {

thread_local std::string g_last_error;

int32_t fail(int32_t code, const std::string &msg) {
    g_last_error = msg;
    return code;
}

#define HIP_TRY(expr)                                                                              \
    do {                                                                                           \
        hipError_t e_ = (expr);                                                                    \
        if (e_ != hipSuccess) return fail(RECMG_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
    } while (0)

constexpr uint32_t kMagic = 0x52434d47u;  // "RCMG"

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

int bitlen(uint64_t x) {
    int b = 0;
    while (x) {
        ++b;
        x >>= 1;
    }
    return b;
}

int64_t pow2ceil(int64_t x) {
    int64_t p = 1;
    while (p < x) p <<= 1;
    return p;
}

#ifndef RECMG_RING_SLACK
#define RECMG_RING_SLACK 3  // resident-ring buffers hold Cap + this many placements' appends (>= 1)
#endif

struct Geom {
    int64_t rows = 0;
    int32_t dim = 0, dtype = 0, esz = 0, row_bytes = 0, cap = 0;
    int64_t map_cap = 0, bm_words = 0;
    int32_t bm_nblk = 0, gsz = 0, nchunk = 0, vec = 0, bpb = 0, copy_unit = 0;
    int32_t wlw = 0, wr = 0, wnch = 0, kind = 0;
    int32_t ways = 0, nsets = 0, qbits = 0;  // set-associative form (ways > 0)
    bool staged = false;                      // misses and fills gathered on the host
    int32_t ring_cap = 0;                     // entries per resident-ring buffer (0: radix select)
};

struct Layout {
    size_t total = 0, host_total = 0;
    std::vector<size_t> pool, slot_row, slot_score, slot_flags, slot_touch, slot_cbit, free_stack, map, bitmap, rank,
        seg, freq, slot_pos, ring0, ring1, rcnt0, rcnt1, roff;
    size_t tabs = 0, st = 0, err = 0, bm_block_start = 0, blocksum = 0, blockoff = 0, tstart = 0, pstart = 0;
    size_t src = 0, raddr = 0, U = 0, slotU = 0, M = 0, mflags = 0, mcbit = 0, mscore = 0, fill_src = 0, fill_slot = 0;
    size_t NP = 0, PU = 0, hist = 0, dump = 0, dump_count = 0, pool_bstart = 0, pool_btab = 0, ftstart = 0;
    size_t sa_bstart = 0, sa_btab = 0, fdesc = 0, stat_log = 0, pfrom = 0, sa_part = 0;
    size_t fstage = 0;
    size_t puref = 0, zone = 0, mslot = 0, npslot = 0, pend_row[2] = {0, 0}, pend_slot[2] = {0, 0};
    // pinned host staging (STAGED): miss ids, miss rows, fill sources, prefetch rows
    size_t h_mrows = 0, h_rows = 0, h_fsrc = 0, h_frows = 0, h_np = 0, h_early = 0;
    size_t staging[2] = {0, 0};
    int64_t stage_stride = 0, sum_cap = 0;
    int32_t total_bm_blocks = 0;
};

int32_t check_config(const recmg_config_t *cfg, std::vector<Geom> *geo) {
    if (!cfg) return fail(RECMG_E_INVALID, "config is NULL");
    const int T = cfg->num_tables;
    if (T < 1 || T > RECMG_MAX_TABLES) return fail(RECMG_E_INVALID, "num_tables out of [1, RECMG_MAX_TABLES]");
    if (!cfg->rows || !cfg->dims || !cfg->dtypes || !cfg->host_tables || !cfg->cache_rows)
        return fail(RECMG_E_INVALID, "a per-table array is NULL");
    if (cfg->policy != RECMG_LRU_BATCH && cfg->policy != RECMG_PRIORITY && cfg->policy != RECMG_LFU_BATCH)
        return fail(RECMG_E_INVALID, "bad policy");
    if (cfg->eviction_speed < 0 || cfg->eviction_speed > (1 << 20))
        return fail(RECMG_E_INVALID, "eviction_speed out of [0, 2^20]");
    if (cfg->miss_mode != RECMG_ZERO_COPY && cfg->miss_mode != RECMG_STAGED) return fail(RECMG_E_INVALID, "bad miss_mode");
    if (cfg->timing < 0 || cfg->timing > 2) return fail(RECMG_E_INVALID, "timing must be 0, 1 or 2");
    if (cfg->ways < 0 || cfg->ways > 64) return fail(RECMG_E_INVALID, "ways out of [0, 64]");
    if (cfg->stats_log_calls < 0) return fail(RECMG_E_INVALID, "negative stats_log_calls");
    if (cfg->max_bags_per_table < 0 || cfg->max_indices < 0 || cfg->max_indices >= (int64_t(1) << 31) ||
        cfg->max_prefetch < 0 || cfg->max_prefetch >= (int64_t(1) << 31))
        return fail(RECMG_E_INVALID, "max_* sizes out of range");
    if ((int64_t)T * cfg->max_bags_per_table >= (int64_t(1) << 31)) return fail(RECMG_E_INVALID, "too many bags");
    geo->assign(T, Geom());
    for (int t = 0; t < T; ++t) {
        Geom &g = (*geo)[t];
        g.rows = cfg->rows[t];
        g.dim = cfg->dims[t];
        g.dtype = cfg->dtypes[t];
        if (g.rows < 1 || g.rows >= (int64_t(1) << 31)) return fail(RECMG_E_INVALID, "rows out of [1, 2^31)");
        if (g.dim < 1 || g.dim > (1 << 16)) return fail(RECMG_E_INVALID, "dim out of [1, 65536]");
        if (g.dtype != RECMG_F32 && g.dtype != RECMG_F16 && g.dtype != RECMG_BF16) return fail(RECMG_E_INVALID, "bad dtype");
        if (cfg->cache_rows[t] < 0) return fail(RECMG_E_INVALID, "negative cache_rows");
        if (!cfg->host_tables[t]) return fail(RECMG_E_INVALID, "host table is NULL");
        const int32_t mode = cfg->miss_modes ? cfg->miss_modes[t] : cfg->miss_mode;
        if (mode != RECMG_ZERO_COPY && mode != RECMG_STAGED) return fail(RECMG_E_INVALID, "bad miss_modes entry");
        g.staged = mode == RECMG_STAGED;
        g.esz = g.dtype == RECMG_F32 ? 4 : 2;
        g.row_bytes = g.dim * g.esz;
        g.cap = (int32_t)std::min<int64_t>(cfg->cache_rows[t], g.rows);
        int64_t bm_bits = g.rows;
        if (cfg->ways > 0) {
            // floor(Cap / W) sets of W ways; the Cap mod W slots left over stay
            // unused, and a table with no set caches nothing (the fully
            // associative path with Cap 0 does exactly that)
            g.nsets = g.cap / cfg->ways;
            g.cap = g.nsets * cfg->ways;
            if (g.nsets > 0) {
                g.ways = cfg->ways;
                g.qbits = bitlen((uint64_t)((g.rows - 1) / g.nsets));
                bm_bits = (int64_t)g.nsets << g.qbits;  // < 2 N_t
            }
        }
        g.map_cap = g.ways ? 64 : pow2ceil(std::max<int64_t>(64, 4 * (int64_t)g.cap));  // load <= 1/4
        const int64_t words = (bm_bits + 31) / 32;
        g.bm_nblk = (int32_t)((words + kWordsPerBlock - 1) / kWordsPerBlock);
        g.bm_words = (int64_t)g.bm_nblk * kWordsPerBlock;
        g.vec = g.row_bytes % 16 == 0;
        if (g.vec && (reinterpret_cast<uintptr_t>(cfg->host_tables[t]) & 15))
            return fail(RECMG_E_INVALID, "host table not 16-byte aligned");
        const int ve = g.vec ? 16 / g.esz : 1;
        const int lanes = (g.dim + ve - 1) / ve;
        g.gsz = (int32_t)std::min<int64_t>(64, std::max<int64_t>(4, pow2ceil(lanes)));
        g.nchunk = (lanes + g.gsz - 1) / g.gsz;
        g.bpb = (kBlock / 64) * (64 / g.gsz);
        // wave-per-bag pooling: rows of 1024 bytes (or whole multiples) are
        // read 64 lanes x 16 bytes per load instruction; 512- and 256-byte
        // rows 2 or 4 to an instruction (16 bytes per lane), 128- and 64-byte
        // rows 4 to an instruction (8 or 4 bytes per lane)
        const int32_t rb = g.row_bytes;
        g.wlw = 0;
        if (rb % 1024 == 0) g.wlw = 16, g.wr = 1, g.wnch = rb / 1024;
        else if (rb == 512) g.wlw = 16, g.wr = 2, g.wnch = 1;
        else if (rb == 256) g.wlw = 16, g.wr = 4, g.wnch = 1;
        else if (rb == 128) g.wlw = 8, g.wr = 4, g.wnch = 1;
        else if (rb == 64) g.wlw = 4, g.wr = 4, g.wnch = 1;
        if (g.wlw) g.bpb = (kBlock / 64) * kWaveBags;
        g.kind = pool_kind(g.dtype, g.vec, g.wlw, g.wr);
        g.copy_unit = g.row_bytes % 16 == 0 ? 16 : (g.row_bytes % 4 == 0 ? 4 : 2);
        // LRU_BATCH fully associative tables keep their residents in key order
        // (ring.hip).  A placement appends at most max_prefetch + max_indices
        // entries; after a compaction at most Cap are live, and the rest of the
        // buffer takes the appends of the placements until the next one.
        const int64_t per_plc = cfg->max_indices + cfg->max_prefetch;
        const int64_t rc = ((int64_t)g.cap + RECMG_RING_SLACK * per_plc + 2 * kRingChunk) / kRingChunk * kRingChunk;
        if (cfg->policy == RECMG_LRU_BATCH && !g.ways && g.cap > 0 && cfg->max_indices < (1 << 30) - 1 &&
            cfg->max_prefetch < (1 << 30) - 1 && cfg->max_indices + 2 * cfg->max_prefetch < (int64_t(1) << 31) &&
            rc < (int64_t(1) << 31) - kRingChunk)
            g.ring_cap = (int32_t)rc;
    }

    return RECMG_OK;
}

bool any_staged(const std::vector<Geom> &geo) {
    for (const Geom &g : geo)
        if (g.staged) return true;
    return false;
}

void make_layout(const recmg_config_t *cfg, const std::vector<Geom> &geo, Layout *L) {
    const int T = (int)geo.size();
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off = align256(off + std::max<size_t>(bytes, 1));
        return at;
    };
    int32_t maxrb = 0;
    bool any_ring = false;
    for (const Geom &g : geo) maxrb = std::max(maxrb, g.row_bytes);
    L->stage_stride = ((int64_t)maxrb + 15) / 16 * 16;
    for (int t = 0; t < T; ++t) {
        const Geom &g = geo[t];
        L->pool.push_back(take((size_t)g.cap * g.row_bytes));
        L->slot_row.push_back(take((size_t)g.cap * 4));
        L->slot_score.push_back(take((size_t)g.cap * 4));
        L->slot_flags.push_back(take((size_t)g.cap * 4));
        L->slot_touch.push_back(take((size_t)g.cap * 4));
        L->slot_cbit.push_back(take((size_t)g.cap));
        L->free_stack.push_back(take((size_t)g.cap * 4));
        L->map.push_back(take((size_t)g.map_cap * 8));
        L->bitmap.push_back(take((size_t)g.bm_words * 4));
        L->rank.push_back(take((size_t)g.bm_words * 16));
        L->seg.push_back(take((size_t)g.nsets * 16));
        L->freq.push_back(take(cfg->policy == RECMG_LFU_BATCH ? (size_t)g.rows * 4 : 0));
        const size_t rc = (size_t)g.ring_cap;
        L->slot_pos.push_back(take(rc ? (size_t)g.cap * 4 : 0));
        L->ring0.push_back(take(rc * 4));
        L->ring1.push_back(take(rc * 4));
        L->rcnt0.push_back(take(rc / kRingChunk * 4));
        L->rcnt1.push_back(take(rc / kRingChunk * 4));
        L->roff.push_back(take(rc / kRingChunk * 4));
        if (rc) any_ring = true;
        L->total_bm_blocks += g.bm_nblk;
        L->sum_cap += g.cap;
    }
    const size_t mi = (size_t)cfg->max_indices, mp = (size_t)cfg->max_prefetch;
    L->tabs = take(sizeof(DTable) * T);
    L->st = take(sizeof(TState) * T);
    L->err = take(4);
    L->bm_block_start = take(4 * (T + 1));
    L->blocksum = take(4 * (size_t)L->total_bm_blocks);
    L->blockoff = take(4 * (size_t)L->total_bm_blocks);
    L->tstart = take(8 * (T + 1));
    L->pstart = take(8 * (T + 1));
    L->src = take(4 * mi);
    L->raddr = take(8 * (mi + kRaddrPad));  // blocks of row addresses are read past the end
    L->U = take(4 * mi);
    L->slotU = take(4 * mi);
    L->M = take(4 * mi);
    L->mflags = take(4 * mi);
    L->mcbit = take(mi);
    L->mscore = take(4 * mi);
    L->NP = take(4 * mp);
    L->PU = take(4 * mp);
    L->fill_src = take(4 * 2 * (mi + mp));   // two fill lists: a placement's fill may still
    L->fill_slot = take(4 * 2 * (mi + mp));  // read one while the next placement writes the other
    L->fdesc = take(8 * 4 * 2 * (size_t)T);
    L->hist = take(4 * (size_t)kRadix * T);
    L->dump = take(4 * (size_t)L->sum_cap);
    L->dump_count = take(4 * T);
    L->pool_bstart = take(4 * (T + 1));
    L->pool_btab = take(4 * T);
    L->ftstart = take(8 * (T + 1));
    L->stat_log = take((size_t)cfg->stats_log_calls * T * sizeof(recmg_table_stats_t));
    L->sa_bstart = take(4 * (T + 1));
    L->sa_btab = take(4 * T);
    L->pfrom = take(cfg->ways > 0 ? 4 * mp : 0);
    int64_t sa_blocks = 0;  // blocks of the set-associative placement (as cache_init counts them)
    for (const Geom &g : geo)
        if (g.ways) sa_blocks += (g.nsets + kSaWaves * sa_sets_per_wave(g.ways, g.nsets) - 1) /
                                 (kSaWaves * sa_sets_per_wave(g.ways, g.nsets));
    L->sa_part = take(8 * 8 * (size_t)sa_blocks);
    L->puref = take(4 * mp);
    L->zone = take(any_ring ? 8 * (mi + mp) : 0);
    L->mslot = take(any_ring ? 4 * mi : 0);
    L->npslot = take(any_ring ? 4 * mp : 0);
    for (int k = 0; k < 2; ++k) {
        L->pend_row[k] = take(any_ring ? 4 * mp : 0);
        L->pend_slot[k] = take(any_ring ? 4 * mp : 0);
    }
    L->staging[0] = take(mi * (size_t)L->stage_stride);
    L->staging[1] = take(mi * (size_t)L->stage_stride);
    const bool staged = any_staged(geo);
    L->fstage = take(staged ? mp * (size_t)L->stage_stride : 0);
    L->total = off;
    if (staged) {
        size_t h = 0;
        auto htake = [&](size_t bytes) {
            const size_t at = h;
            h = align256(h + std::max<size_t>(bytes, 1));
            return at;
        };
        L->h_mrows = htake(4 * mi);
        L->h_rows = htake(mi * (size_t)L->stage_stride);
        L->h_fsrc = htake(4 * (mi + mp));
        L->h_frows = htake(mp * (size_t)L->stage_stride);
        L->h_np = htake(4 * mp);
        L->h_early = htake(sizeof(TState) * T + 8 * (T + 1) + 8);
        L->host_total = h;
    }
}

}  // namespace

struct recmg_cache {
    uint32_t magic = kMagic;
    int device = 0;
    int T = 0;
    recmg_config_t cfg{};
    std::vector<Geom> geo;
    Layout L;
    DGlobal g{};
    std::vector<const char *> host;  // host tables (host pointers)
    int32_t max_cap = 0, max_map = 0, max_units = 0, rowbits = 1, nsa = 0, max_nblk = 0;
    int64_t sa_blocks = 0;   // blocks of the set-associative placement kernel
    int64_t sa_blocks1 = 0;  // the first of them, over the tables of one set per wave
    int64_t sa_max_blocks = 0;  // the most blocks of one table
    bool has_fa = false, has_sa = false;  // tables of each form present
    bool has_ring = false, has_scan_fa = false;  // fully associative tables with and without a resident ring
    int32_t max_ring_chunks = 0;
    bool has_zc = false, has_staged = false;  // tables of each miss mode present
    std::vector<int32_t> pool_order;  // table ids ordered by pooled-kernel kind
    std::vector<PoolLaunch> pool_launches;
    int64_t max_rows = 0;
    int64_t placements = 0, forwards = 0, last_n = 0;
    int64_t calls = 0;  // placements + forwards so far (the stats log's call index)
    bool have_fwd = false;
    hipStream_t last_stream = nullptr;
    // Calls may come on different streams (e.g. the next placement on its own
    // stream while the last forward still runs): each call waits for what it
    // needs from the latest call of the other kind through these events.
    hipStream_t fwd_stream = nullptr, plc_stream = nullptr;
    bool fwd_ev = false, plc_ev = false;  // the events below were recorded
    hipEvent_t ev_src = nullptr;   // latest forward: after its dedup, probe, sources and coverage
    hipEvent_t ev_pool = nullptr;  // latest forward: after its pooled kernel
    hipEvent_t ev_fwd = nullptr;   // latest forward: after all its kernels
    hipEvent_t ev_plc = nullptr;   // latest placement: after all its kernels but the fill
    hipEvent_t ev_fill[2] = {nullptr, nullptr};  // fill of the latest placement of each parity
    bool fill_rec[2] = {false, false};
    hipStream_t fill_stream[2] = {nullptr, nullptr};  // stream each parity's latest fill ran on
    int fill_last = -1;  // parity of the latest fill no forward has waited for yet
    // An error after a call began enqueuing work leaves device and host state
    // out of step: every later call but destroy is refused.
    bool broken = false;
    bool static_ws = false;  // the workspace is the device's static array (recmg_cache_init_static)
    int32_t *fill_src_buf[2] = {nullptr, nullptr}, *fill_slot_buf[2] = {nullptr, nullptr};
    int64_t *fdesc_buf[2] = {nullptr, nullptr};
    int32_t pool_B = -1;
    int64_t plc_np = -1;  // prefetch ids of the placement since the last forward (-1: none)
    int64_t plc_np_last = 0;  // prefetch ids of the latest placement
    char *stage[2] = {nullptr, nullptr};  // staging buffers, alternating between forwards
    int cur = 0;                          // buffer of the latest forward

    int64_t pool_blocks = 0;
    std::vector<int32_t> pool_bstart;
    // STAGED
    hipStream_t copy_stream = nullptr;
    hipEvent_t ev_ready = nullptr, ev_copied = nullptr;
    hipEvent_t ev_np = nullptr;  // a placement's new prefetch candidates have reached the host
    int32_t *h_np = nullptr;     // those candidates (NP), for the early gather
    // pinned copies made with them: table states, prefetch list starts, error word
    TState *he_st = nullptr;
    int64_t *he_pstart = nullptr;
    int32_t *he_err = nullptr;
    bool has_staged_fa = false;  // STAGED fully associative tables with slots (gathered early)
    bool has_staged_sa = false;  // STAGED set-associative tables (gathered after their placement)
    int32_t *h_mrows = nullptr;
    char *h_rows = nullptr;
    int32_t *h_fsrc = nullptr;  // fill sources of a placement, rewritten to staged rows
    char *h_frows = nullptr;    // prefetch rows gathered on the host
    std::vector<int64_t> h_pstart, h_ftstart;
    std::vector<TState> h_st;
    std::vector<int64_t> h_tstart;
    // stage timing: 0 off, 1 the pooled kernel only, 2 every stage
    int32_t timing = 0;
    struct Mark {
        int stage;
        hipEvent_t a, b;
    };
    std::vector<hipEvent_t> ev_free;
    std::vector<Mark> marks;
    double stage_ms[RECMG_NUM_STAGES] = {0};
    int64_t stage_calls[RECMG_NUM_STAGES] = {0};

    // Every event the handle created, also when init stops half way.  The
    // caller of delete has synchronised (or nothing was enqueued).
    ~recmg_cache() {
        for (hipEvent_t e : {ev_src, ev_pool, ev_fwd, ev_plc, ev_fill[0], ev_fill[1], ev_ready, ev_copied, ev_np})
            if (e) (void)hipEventDestroy(e);
        for (const Mark &m : marks) {
            if (m.a) (void)hipEventDestroy(m.a);
            if (m.b) (void)hipEventDestroy(m.b);
        }
        for (hipEvent_t e : ev_free)
            if (e) (void)hipEventDestroy(e);
    }
};

namespace {

hipEvent_t take_event(recmg_cache_t *c);

// Timing level 1: an event pair that the kernel's own dispatch records (no
// stream command is added), kept as a mark of `stage` once the launch is
// issued.  Both null when not timing at level 1 or out of events.
struct DispatchTimer {
    recmg_cache_t *c;
    int stage;
    hipEvent_t a = nullptr, b = nullptr;
    DispatchTimer(recmg_cache_t *c_, int stage_, bool on);
    void issued();
    ~DispatchTimer();
};

hipEvent_t take_event(recmg_cache_t *c) {
    if (c->ev_free.empty()) {
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        return e;
    }
    hipEvent_t e = c->ev_free.back();
    c->ev_free.pop_back();
    return e;
}

DispatchTimer::DispatchTimer(recmg_cache_t *c_, int stage_, bool on) : c(c_), stage(stage_) {
    if (!on || c->timing != 1) return;
    a = take_event(c);
    b = a ? take_event(c) : nullptr;
    if (a && !b) {
        c->ev_free.push_back(a);
        a = nullptr;
    }
}
void DispatchTimer::issued() {
    if (a) c->marks.push_back({stage, a, b});
    a = b = nullptr;
}
DispatchTimer::~DispatchTimer() {  // not issued: the events go back unused
    if (a) c->ev_free.push_back(a);
    if (b) c->ev_free.push_back(b);
}

// Stage timing (level 2): an event pair per stage per call, resolved in
// recmg_stage_times.  Each pair adds two commands to the stream (a few us).
struct StageTimer {
    recmg_cache_t *c;
    int stage;
    hipStream_t s;
    hipEvent_t a = nullptr;
    StageTimer(recmg_cache_t *c_, int stage_, hipStream_t s_) : c(c_), stage(stage_), s(s_) {
        if (c->timing < 2) return;
        a = take();
        if (a) (void)hipEventRecord(a, s);
    }
    hipEvent_t take() { return take_event(c); }
    ~StageTimer() {
        if (!a) return;
        hipEvent_t b = take();
        if (!b) {
            c->ev_free.push_back(a);
            return;
        }
        (void)hipEventRecord(b, s);
        c->marks.push_back({stage, a, b});
    }
};

int32_t check_handle(recmg_cache_t *c) {
    if (!c) return fail(RECMG_E_INVALID, "handle is NULL");
    if (c->magic != kMagic) return fail(RECMG_E_STATE, "handle is not live");
    if (c->broken)
        return fail(RECMG_E_STATE, "an earlier call failed after enqueuing work; the handle must be destroyed");
    return RECMG_OK;
}

// Marks the handle broken unless the call reaches its end: errors returned
// once a call has started enqueuing device work leave the device state ahead
// of the host bookkeeping.
struct EnqueueGuard {
    recmg_cache_t *c;
    bool done = false;
    explicit EnqueueGuard(recmg_cache_t *c_) : c(c_) {}
    ~EnqueueGuard() {
        if (!done) c->broken = true;
    }
};

// Waits for every stream the handle's calls used.
hipError_t sync_all(recmg_cache_t *c) {
    hipError_t e = hipStreamSynchronize(c->last_stream);
    if (e == hipSuccess && c->fwd_ev) e = hipStreamSynchronize(c->fwd_stream);
    if (e == hipSuccess && c->plc_ev) e = hipStreamSynchronize(c->plc_stream);
    if (e == hipSuccess && c->copy_stream) e = hipStreamSynchronize(c->copy_stream);
    if (e == hipSuccess) c->fill_last = -1;
    return e;
}

int32_t set_device(recmg_cache_t *c) {
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur));
    if (cur != c->device) HIP_TRY(hipSetDevice(c->device));
    return RECMG_OK;
}

// Host gather for the STAGED paths.  Each table's list of n[t] rows is cut
// into chunks of kChunk rows, and consecutive chunks into copy groups of
// kGroup rows.  Worker threads gather chunks in order; the calling thread
// issues a group's copies to the device as soon as all its chunks are done,
// so the gather and the host-to-device copies overlap.
constexpr int64_t kChunk = 2048, kGroup = 16384;
// Rows are scattered over the tables, so each is a cache and TLB miss; the
// gather loops touch the row kAhead entries ahead to keep several in flight.
constexpr int64_t kAhead = 12;

inline void prefetch_row(const char *p, int64_t bytes) {
    for (int64_t o = 0; o < bytes; o += 64) __builtin_prefetch(p + o, 0, 0);
}

template <class Work, class Copy>
int32_t gather_and_copy(const std::vector<int64_t> &n, Work work, Copy copy) {
    struct Chunk {
        int t;
        int64_t lo, hi;
        int group;
    };
    struct Group {
        int t;
        int64_t lo, hi;
        int nchunks;
    };
    std::vector<Chunk> chunks;
    std::vector<Group> groups;
    for (int t = 0; t < (int)n.size(); ++t)
        for (int64_t g0 = 0; g0 < n[t]; g0 += kGroup) {
            const int64_t g1 = std::min(n[t], g0 + kGroup);
            groups.push_back({t, g0, g1, 0});
            for (int64_t c0 = g0; c0 < g1; c0 += kChunk) {
                chunks.push_back({t, c0, std::min(g1, c0 + kChunk), (int)groups.size() - 1});
                groups.back().nchunks++;
            }
        }
    if (chunks.empty()) return RECMG_OK;
    std::unique_ptr<std::atomic<int>[]> done(new std::atomic<int>[groups.size()]);
    for (size_t k = 0; k < groups.size(); ++k) done[k].store(0);
    std::atomic<size_t> next(0);
    const unsigned hw = std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
    const unsigned nth = (unsigned)std::min<size_t>(hw, chunks.size());
    std::vector<std::thread> th;
    for (unsigned k = 0; k < nth; ++k)
        th.emplace_back([&] {
            for (size_t i; (i = next.fetch_add(1)) < chunks.size();) {
                work(chunks[i].t, chunks[i].lo, chunks[i].hi);
                done[chunks[i].group].fetch_add(1, std::memory_order_release);
            }
        });
    int32_t rc = RECMG_OK;
    for (size_t k = 0; k < groups.size(); ++k) {
        while (done[k].load(std::memory_order_acquire) < groups[k].nchunks) std::this_thread::yield();
        if (rc == RECMG_OK) rc = copy(groups[k].t, groups[k].lo, groups[k].hi);
    }
    for (auto &x : th) x.join();
    return rc;
}

// STAGED prefetch fill: the fill list comes back to the host, the host
// gathers the prefetch rows from its tables into pinned staging and rewrites
// their sources to staged rows, copies move both to the device on stream cs,
// and the fill kernel (launched by the caller on cs) copies rows into slots.
int32_t staged_fill(recmg_cache_t *c, hipStream_t s, hipStream_t cs) {
    const int T = c->T;
    HIP_TRY(hipMemcpyAsync(c->h_st.data(), c->g.st, sizeof(TState) * T, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(c->h_pstart.data(), c->g.pstart, 8 * (T + 1), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(c->h_ftstart.data(), c->g.ftstart, 8 * (T + 1), hipMemcpyDeviceToHost, s));
    int32_t err = 0;
    HIP_TRY(hipMemcpyAsync(&err, c->g.err, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (err) return RECMG_OK;
    std::vector<int64_t> base(T), nfill(T, 0);
    int64_t total = 0;
    for (int t = 0; t < T; ++t) {
        base[t] = c->h_ftstart[t] + c->h_pstart[t];
        // zero-copy tables' fills read the host themselves; fully associative
        // STAGED tables' prefetch rows were gathered early (early_gather)
        nfill[t] = c->geo[t].staged && c->geo[t].ways ? c->h_st[t].popped : 0;
        if (base[t] < 0 || nfill[t] < 0 || base[t] + nfill[t] > c->g.fill_cap)
            return fail(RECMG_E_STATE, "fill list outside its buffer");
        if (nfill[t])
            HIP_TRY(hipMemcpyAsync(c->h_fsrc + base[t], c->g.fill_src + base[t], 4 * (size_t)nfill[t],
                                   hipMemcpyDeviceToHost, s));
        total += nfill[t];
    }
    if (total == 0) return RECMG_OK;
    HIP_TRY(hipStreamSynchronize(s));
    const int64_t stride = c->L.stage_stride;
    // host-sourced entries are packed in list order: chunk k of table t starts
    // at kbase[t][k] among them
    std::vector<std::vector<int64_t>> kbase(T);
    for (int t = 0; t < T; ++t) {
        const int64_t nck = (nfill[t] + kChunk - 1) / kChunk;
        kbase[t].assign(nck + 1, 0);
        for (int64_t k = 0; k < nck; ++k) {
            int64_t cnt = 0;
            for (int64_t j = k * kChunk; j < std::min(nfill[t], (k + 1) * kChunk); ++j) cnt += c->h_fsrc[base[t] + j] < 0;
            kbase[t][k + 1] = kbase[t][k] + cnt;
        }
        if (kbase[t][nck] > c->h_pstart[t + 1] - c->h_pstart[t])
            return fail(RECMG_E_STATE, "staged fills exceed the list");
    }
    auto work = [&](int t, int64_t lo, int64_t hi) {
        const int64_t rb = c->geo[t].row_bytes, p0 = c->h_pstart[t];
        int64_t k = kbase[t][lo / kChunk];
        for (int64_t j = lo; j < hi; ++j) {
            if (j + kAhead < hi && c->h_fsrc[base[t] + j + kAhead] < 0)
                prefetch_row(c->host[t] + (-(int64_t)c->h_fsrc[base[t] + j + kAhead] - 1) * rb, rb);
            int32_t &src = c->h_fsrc[base[t] + j];
            if (src >= 0) continue;  // an admitted miss: already in HBM staging
            const int64_t row = -(int64_t)src - 1;
            std::memcpy(c->h_frows + (p0 + k) * stride, c->host[t] + row * rb, (size_t)rb);
            src = -(int32_t)(p0 + k) - 1;  // now: staged prefetch row p0 + k
            ++k;
        }
    };
    auto copy = [&](int t, int64_t lo, int64_t hi) -> int32_t {
        HIP_TRY(hipMemcpyAsync(c->g.fill_src + base[t] + lo, c->h_fsrc + base[t] + lo, 4 * (size_t)(hi - lo),
                               hipMemcpyHostToDevice, cs));
        const int64_t k0 = kbase[t][lo / kChunk], k1 = kbase[t][(hi + kChunk - 1) / kChunk];
        const int64_t r0 = c->h_pstart[t] + k0;
        if (k1 > k0)
            HIP_TRY(hipMemcpyAsync(c->g.fstage + r0 * stride, c->h_frows + r0 * stride, (size_t)((k1 - k0) * stride),
                                   hipMemcpyHostToDevice, cs));
        return RECMG_OK;
    };
    return gather_and_copy(nfill, work, copy);
}

// Early gather of the prefetch rows of fully associative STAGED tables: the
// placement's new prefetch candidates (NP, with their counts) came back to
// the host right after classification (ev_np), so the host gathers their rows
// into pinned staging and copies them to the device (fstage row pstart[t] + k
// for NP[pstart[t] + k]) while the GPU ranks and admits; admission points each
// admitted candidate's fill at that row.  A candidate the ranking drops was
// gathered for nothing (under LRU a new prefetch candidate is dropped only
// when the candidates outnumber the cache).
int32_t early_gather(recmg_cache_t *c, hipStream_t cs) {
    const int T = c->T;
    HIP_TRY(hipEventSynchronize(c->ev_np));
    if (*c->he_err) return RECMG_OK;  // the device flag already disables the rest
    const int64_t *ps = c->he_pstart;
    std::vector<int64_t> n(T, 0);
    for (int t = 0; t < T; ++t) {
        const Geom &ge = c->geo[t];
        if (!ge.staged || ge.ways || ge.cap == 0) continue;
        n[t] = c->he_st[t].npcount;
        if (n[t] < 0 || ps[t] < 0 || ps[t] + n[t] > ps[t + 1] || ps[t + 1] > c->cfg.max_prefetch)
            return fail(RECMG_E_STATE, "prefetch candidates outside their list");
    }
    const int64_t stride = c->L.stage_stride;
    auto work = [&](int t, int64_t lo, int64_t hi) {
        const int64_t p0 = ps[t], rb = c->geo[t].row_bytes;
        for (int64_t k = lo; k < hi; ++k) {
            if (k + kAhead < hi) prefetch_row(c->host[t] + (int64_t)c->h_np[p0 + k + kAhead] * rb, rb);
            std::memcpy(c->h_frows + (p0 + k) * stride, c->host[t] + (int64_t)c->h_np[p0 + k] * rb, (size_t)rb);
        }
    };
    auto copy = [&](int t, int64_t lo, int64_t hi) -> int32_t {
        const int64_t r0 = ps[t] + lo;
        HIP_TRY(hipMemcpyAsync(c->g.fstage + r0 * stride, c->h_frows + r0 * stride, (size_t)((hi - lo) * stride),
                               hipMemcpyHostToDevice, cs));
        return RECMG_OK;
    };
    return gather_and_copy(n, work, copy);
}

// STAGED miss path: miss ids of the STAGED tables to the host, a parallel
// host gather into pinned staging overlapped with the copies on the copy
// stream; the compute stream waits for the copies.  The zero-copy tables'
// misses are fetched by the kernel, launched once the host has read what it
// needs (so that its waits do not wait for the kernel), beside the gather.
int32_t staged_fetch(recmg_cache_t *c, hipStream_t s) {
    const int T = c->T;
    HIP_TRY(hipMemcpyAsync(c->h_st.data(), c->g.st, sizeof(TState) * T, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipMemcpyAsync(c->h_tstart.data(), c->g.tstart, 8 * (T + 1), hipMemcpyDeviceToHost, s));
    int32_t err = 0;
    HIP_TRY(hipMemcpyAsync(&err, c->g.err, 4, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    auto zero_copy_fetch = [&]() -> int32_t {
        if (c->has_zc) {
            DispatchTimer dt(c, RECMG_STAGE_FWD_FETCH, true);
            launch_fetch(c->g, s, dt.a, dt.b);
            dt.issued();
        }
        return RECMG_OK;
    };
    if (err) return zero_copy_fetch();  // the device flag already disables the rest
    std::vector<int64_t> nm(T);
    int64_t total = 0;
    for (int t = 0; t < T; ++t) {
        nm[t] = c->geo[t].staged ? c->h_st[t].mcount : 0;
        if (nm[t])
            HIP_TRY(hipMemcpyAsync(c->h_mrows + c->h_tstart[t], c->g.M + c->h_tstart[t], 4 * (size_t)nm[t],
                                   hipMemcpyDeviceToHost, s));
        total += nm[t];
    }
    if (total == 0) return zero_copy_fetch();
    HIP_TRY(hipStreamSynchronize(s));
    const int64_t stride = c->L.stage_stride;
    hipStream_t cs = c->copy_stream ? c->copy_stream : s;
    if (cs != s) {
        HIP_TRY(hipEventRecord(c->ev_ready, s));
        HIP_TRY(hipStreamWaitEvent(cs, c->ev_ready, 0));
    }
    if ((err = zero_copy_fetch())) return err;
    auto work = [&](int t, int64_t lo, int64_t hi) {
        const int64_t ts = c->h_tstart[t], rb = c->geo[t].row_bytes;
        for (int64_t m = lo; m < hi; ++m) {
            if (m + kAhead < hi) prefetch_row(c->host[t] + (int64_t)c->h_mrows[ts + m + kAhead] * rb, rb);
            std::memcpy(c->h_rows + (ts + m) * stride, c->host[t] + (int64_t)c->h_mrows[ts + m] * rb, (size_t)rb);
        }
    };
    auto copy = [&](int t, int64_t lo, int64_t hi) -> int32_t {
        const int64_t r0 = c->h_tstart[t] + lo;
        HIP_TRY(hipMemcpyAsync(c->g.staging + r0 * stride, c->h_rows + r0 * stride, (size_t)((hi - lo) * stride),
                               hipMemcpyHostToDevice, cs));
        return RECMG_OK;
    };
    int32_t rc = gather_and_copy(nm, work, copy);
    if (rc) return rc;
    if (cs != s) {
        HIP_TRY(hipEventRecord(c->ev_copied, cs));
        HIP_TRY(hipStreamWaitEvent(s, c->ev_copied, 0));
    }
    return RECMG_OK;
}

int32_t host_check_ids(const int32_t *dev_ids, const int64_t *dev_off, int64_t n_off, int64_t stride_off,
                       int64_t n_ids, const std::vector<Geom> &geo, hipStream_t s) {
    std::vector<int64_t> off(n_off);
    std::vector<int32_t> ids(std::max<int64_t>(n_ids, 1));
    HIP_TRY(hipMemcpyAsync(off.data(), dev_off, 8 * n_off, hipMemcpyDeviceToHost, s));
    if (n_ids > 0) HIP_TRY(hipMemcpyAsync(ids.data(), dev_ids, 4 * n_ids, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (off[0] != 0 || off[n_off - 1] != n_ids) return fail(RECMG_E_RANGE, "offsets do not span the ids");
    for (int64_t i = 0; i + 1 < n_off; ++i)
        if (off[i] > off[i + 1]) return fail(RECMG_E_RANGE, "offsets decrease");
    for (size_t t = 0; t < geo.size(); ++t)
        for (int64_t i = off[t * stride_off]; i < off[(t + 1) * stride_off]; ++i)
            if (ids[i] < 0 || ids[i] >= geo[t].rows) return fail(RECMG_E_RANGE, "row id out of range");
    return RECMG_OK;
}

// Workspace of the handles recmg_cache_init_static makes, for callers that
// cannot allocate device memory: a fixed array in the library's code object,
// one copy per device, held until the process ends.  Host code never uses the
// array's name as an address (it is a host-side stand-in there): the device
// address comes from hipGetSymbolAddress, once per device.
constexpr size_t kStaticWorkspaceBytes = size_t(32) << 20;
static __device__ __align__(256) unsigned char scratch[kStaticWorkspaceBytes];

constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
void *g_static_ptr[kMaxDevices];              // device address of `scratch` per device, set on first use
recmg_cache_t *g_static_owner[kMaxDevices];   // the live handle that holds it, if any

int32_t cache_init(const recmg_config_t *cfg, recmg_cache_t **out);

}  // namespace

extern "C" {

const char *recmg_last_error(void) { return g_last_error.c_str(); }

int32_t recmg_query_workspace(const recmg_config_t *cfg, size_t *device_bytes, size_t *host_staging_bytes) {
    std::vector<Geom> geo;
    int32_t rc = check_config(cfg, &geo);
    if (rc) return rc;
    Layout L;
    make_layout(cfg, geo, &L);
    if (device_bytes) *device_bytes = L.total;
    if (host_staging_bytes) *host_staging_bytes = L.host_total;
    return RECMG_OK;
}

int32_t recmg_cache_init(const recmg_config_t *cfg, recmg_cache_t **out) { return cache_init(cfg, out); }

int32_t recmg_cache_init_static(const recmg_config_t *cfg, recmg_cache_t **out) {
    if (!out) return fail(RECMG_E_INVALID, "out is NULL");
    std::vector<Geom> geo;
    int32_t rc = check_config(cfg, &geo);
    if (rc) return rc;
    Layout L;
    make_layout(cfg, geo, &L);
    if (L.total > kStaticWorkspaceBytes)
        return fail(RECMG_E_NOMEM, "the configuration needs a " + std::to_string(L.total) +
                                       "-byte workspace; the static workspace holds " +
                                       std::to_string(kStaticWorkspaceBytes) + " bytes");
    int dev = -1;
    HIP_TRY(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(RECMG_E_INVALID, "device id beyond the static workspace table");
    std::lock_guard<std::mutex> lock(g_static_mu);
    if (g_static_owner[dev]) return fail(RECMG_E_STATE, "the static workspace of this device is held by a live handle");
    if (!g_static_ptr[dev]) {
        void *p = nullptr;
        HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(RECMG_E_HIP, "hipGetSymbolAddress gave no address for the static workspace");
        g_static_ptr[dev] = p;
    }
    recmg_config_t c2 = *cfg;
    c2.device_workspace = g_static_ptr[dev];
    c2.device_workspace_bytes = kStaticWorkspaceBytes;
    recmg_cache_t *h = nullptr;
    if ((rc = cache_init(&c2, &h))) return rc;
    h->static_ws = true;
    g_static_owner[dev] = h;
    *out = h;
    return RECMG_OK;
}

}  // extern "C"

namespace {

int32_t cache_init(const recmg_config_t *cfg, recmg_cache_t **out) {
    if (!out) return fail(RECMG_E_INVALID, "out is NULL");
    std::vector<Geom> geo;
    int32_t rc = check_config(cfg, &geo);
    if (rc) return rc;
    Layout L;
    make_layout(cfg, geo, &L);
    if (!cfg->device_workspace || cfg->device_workspace_bytes < L.total)
        return fail(RECMG_E_NOMEM, "device workspace smaller than recmg_query_workspace");
    if (reinterpret_cast<uintptr_t>(cfg->device_workspace) & 255)
        return fail(RECMG_E_INVALID, "device workspace not 256-byte aligned");
    if (any_staged(geo) && (!cfg->host_staging || cfg->host_staging_bytes < L.host_total))
        return fail(RECMG_E_NOMEM, "host staging smaller than recmg_query_workspace");
    const int T = cfg->num_tables;

    std::unique_ptr<recmg_cache> c(new recmg_cache());
    HIP_TRY(hipGetDevice(&c->device));
    c->T = T;
    c->cfg = *cfg;
    c->cfg.miss_modes = nullptr;  // the caller's array is read during init only (modes are in geo)
    c->timing = cfg->timing;
    c->geo = geo;
    c->L = L;
    // host tables: must be pinned memory visible to the device
    std::vector<const char *> dev_host(T);
    for (int t = 0; t < T; ++t) {
        c->host.push_back(static_cast<const char *>(cfg->host_tables[t]));
        if (geo[t].staged) c->has_staged = true;
        else c->has_zc = true;
        if (geo[t].staged && geo[t].ways) c->has_staged_sa = true;
        if (geo[t].staged && !geo[t].ways && geo[t].cap > 0) c->has_staged_fa = true;
        if (geo[t].staged) {
            dev_host[t] = nullptr;  // only the host reads the tables: any host memory will do
            continue;
        }
        void *dp = nullptr;
        if (hipHostGetDevicePointer(&dp, const_cast<void *>(cfg->host_tables[t]), 0) != hipSuccess || !dp) {
            (void)hipGetLastError();
            return fail(RECMG_E_INVALID, "host table " + std::to_string(t) + " is not pinned host memory");
        }
        dev_host[t] = static_cast<const char *>(dp);
    }
    char *ws = static_cast<char *>(cfg->device_workspace);
    DGlobal &g = c->g;
    g.tabs = reinterpret_cast<DTable *>(ws + L.tabs);
    g.st = reinterpret_cast<TState *>(ws + L.st);
    g.err = reinterpret_cast<int32_t *>(ws + L.err);
    g.bm_block_start = reinterpret_cast<int32_t *>(ws + L.bm_block_start);
    g.blocksum = reinterpret_cast<int32_t *>(ws + L.blocksum);
    g.blockoff = reinterpret_cast<int32_t *>(ws + L.blockoff);
    g.tstart = reinterpret_cast<int64_t *>(ws + L.tstart);
    g.pstart = reinterpret_cast<int64_t *>(ws + L.pstart);
    g.src = reinterpret_cast<int32_t *>(ws + L.src);
    g.raddr = reinterpret_cast<uint64_t *>(ws + L.raddr);
    g.U = reinterpret_cast<int32_t *>(ws + L.U);
    g.slotU = reinterpret_cast<int32_t *>(ws + L.slotU);
    g.M = reinterpret_cast<int32_t *>(ws + L.M);
    g.mflags = reinterpret_cast<uint32_t *>(ws + L.mflags);
    g.mcbit = reinterpret_cast<uint8_t *>(ws + L.mcbit);
    g.mscore = reinterpret_cast<int32_t *>(ws + L.mscore);
    g.NP = reinterpret_cast<int32_t *>(ws + L.NP);
    g.PU = reinterpret_cast<int32_t *>(ws + L.PU);
    g.ftstart = reinterpret_cast<int64_t *>(ws + L.ftstart);
    for (int k = 0; k < 2; ++k) {
        c->fill_src_buf[k] = reinterpret_cast<int32_t *>(ws + L.fill_src) + k * (cfg->max_indices + cfg->max_prefetch);
        c->fill_slot_buf[k] = reinterpret_cast<int32_t *>(ws + L.fill_slot) + k * (cfg->max_indices + cfg->max_prefetch);
        c->fdesc_buf[k] = reinterpret_cast<int64_t *>(ws + L.fdesc) + k * 4 * T;
    }
    g.fill_src = c->fill_src_buf[0];
    g.fill_slot = c->fill_slot_buf[0];
    g.fill_cap = cfg->max_indices + cfg->max_prefetch;
    g.fstage = ws + L.fstage;
    g.staged_fill = c->has_staged ? 1 : 0;
    g.hist = reinterpret_cast<int32_t *>(ws + L.hist);
    g.dump = reinterpret_cast<int32_t *>(ws + L.dump);
    g.dump_count = reinterpret_cast<int32_t *>(ws + L.dump_count);
    c->stage[0] = ws + L.staging[0];
    c->stage[1] = ws + L.staging[1];
    g.staging = c->stage[0];
    g.stage_stride = L.stage_stride;
    g.T = T;
    g.total_bm_blocks = L.total_bm_blocks;
    g.own_tables = 0;
    g.own_slices = 0;
    g.stat_log = reinterpret_cast<int64_t *>(ws + L.stat_log);
    g.sa_bstart = reinterpret_cast<int32_t *>(ws + L.sa_bstart);
    g.sa_btab = reinterpret_cast<int32_t *>(ws + L.sa_btab);
    g.sa_part = reinterpret_cast<int64_t *>(ws + L.sa_part);
    g.pfrom = reinterpret_cast<int32_t *>(ws + L.pfrom);
    g.puref = reinterpret_cast<int32_t *>(ws + L.puref);
    g.zone = reinterpret_cast<int2 *>(ws + L.zone);
    g.mslot = reinterpret_cast<int32_t *>(ws + L.mslot);
    g.npslot = reinterpret_cast<int32_t *>(ws + L.npslot);
    for (int k = 0; k < 2; ++k) {
        g.pend_row[k] = reinterpret_cast<int32_t *>(ws + L.pend_row[k]);
        g.pend_slot[k] = reinterpret_cast<int32_t *>(ws + L.pend_slot[k]);
    }

    std::vector<DTable> tabs(T);
    std::vector<int32_t> bstart(T + 1, 0);
    int64_t out_off = 0, cap_off = 0;
    for (int t = 0; t < T; ++t) {
        const Geom &ge = geo[t];
        DTable &d = tabs[t];
        std::memset(&d, 0, sizeof(d));
        d.host = dev_host[t];
        d.pool = ws + L.pool[t];
        d.slot_row = reinterpret_cast<int32_t *>(ws + L.slot_row[t]);
        d.slot_score = reinterpret_cast<int32_t *>(ws + L.slot_score[t]);
        d.slot_flags = reinterpret_cast<uint32_t *>(ws + L.slot_flags[t]);
        d.slot_touch = reinterpret_cast<int32_t *>(ws + L.slot_touch[t]);
        d.slot_cbit = reinterpret_cast<uint8_t *>(ws + L.slot_cbit[t]);
        d.free_stack = reinterpret_cast<int32_t *>(ws + L.free_stack[t]);
        d.map = reinterpret_cast<int2 *>(ws + L.map[t]);
        d.bitmap = reinterpret_cast<uint32_t *>(ws + L.bitmap[t]);
        d.rank = reinterpret_cast<uint4 *>(ws + L.rank[t]);
        d.rows = ge.rows;
        d.out_elem_off = out_off;
        d.cap_off = cap_off;
        d.dim = ge.dim;
        d.dtype = ge.dtype;
        d.row_bytes = ge.row_bytes;
        d.cap = ge.cap;
        d.map_mask = (int32_t)(ge.map_cap - 1);
        d.bm_words = (int32_t)ge.bm_words;
        d.bm_block0 = bstart[t];
        d.bm_nblk = ge.bm_nblk;
        d.gsz = ge.gsz;
        d.nchunk = ge.nchunk;
        d.vec = ge.vec;
        d.bags_per_block = ge.bpb;
        d.copy_unit = ge.copy_unit;
        d.wlw = ge.wlw;
        d.wr = ge.wr;
        d.wnch = ge.wnch;
        d.ways = ge.ways;
        d.nsets = ge.ways ? ge.nsets : 0;
        d.qbits = ge.qbits;
        d.staged = ge.staged ? 1 : 0;
        d.seg = reinterpret_cast<int4 *>(ws + L.seg[t]);
        d.freq = cfg->policy == RECMG_LFU_BATCH ? reinterpret_cast<int32_t *>(ws + L.freq[t]) : nullptr;
        if (ge.ring_cap) {
            d.slot_pos = reinterpret_cast<int32_t *>(ws + L.slot_pos[t]);
            d.ring[0] = reinterpret_cast<int32_t *>(ws + L.ring0[t]);
            d.ring[1] = reinterpret_cast<int32_t *>(ws + L.ring1[t]);
            d.rcnt[0] = reinterpret_cast<int32_t *>(ws + L.rcnt0[t]);
            d.rcnt[1] = reinterpret_cast<int32_t *>(ws + L.rcnt1[t]);
            d.roff = reinterpret_cast<int32_t *>(ws + L.roff[t]);
            d.ring_cap = ge.ring_cap;
            c->has_ring = true;
            c->max_ring_chunks = std::max(c->max_ring_chunks, ge.ring_cap / kRingChunk);
        } else if (!ge.ways) {
            c->has_scan_fa = true;
        }
        if (ge.ways) c->has_sa = true;
        else c->has_fa = true;

        bstart[t + 1] = bstart[t] + ge.bm_nblk;
        out_off += ge.dim;
        cap_off += ge.cap;
        c->max_cap = std::max(c->max_cap, ge.cap);
        c->max_map = (int32_t)std::max<int64_t>(c->max_map, ge.map_cap);
        c->max_units = std::max(c->max_units, ge.row_bytes / ge.copy_unit);
        c->max_rows = std::max(c->max_rows, ge.rows);
        c->max_nblk = std::max(c->max_nblk, ge.bm_nblk);
        if (owns_bitmap(ge.bm_nblk)) {
            g.own_tables += 1;
            g.own_slices = std::max(g.own_slices, (ge.bm_nblk + kOwnSliceBlocks - 1) / kOwnSliceBlocks);
        }
    }
    c->rowbits = std::max(1, bitlen((uint64_t)(c->max_rows - 1)));
    c->pool_order.resize(T);
    for (int t = 0; t < T; ++t) c->pool_order[t] = t;
    std::stable_sort(c->pool_order.begin(), c->pool_order.end(),
                     [&](int x, int y) { return geo[x].kind < geo[y].kind; });
    // set-associative placement: tables with the fewest sets first, kSaWaves
    // waves of sa_sets_per_wave(ways, nsets) sets each per block
    std::vector<int32_t> sa_tab, sa_bs(1, 0);
    for (int t = 0; t < T; ++t)
        if (geo[t].ways) sa_tab.push_back(t);
    std::stable_sort(sa_tab.begin(), sa_tab.end(), [&](int x, int y) { return geo[x].nsets < geo[y].nsets; });
    for (int t : sa_tab) {
        const int spw = sa_sets_per_wave(geo[t].ways, geo[t].nsets);
        const int per_block = kSaWaves * spw;
        sa_bs.push_back(sa_bs.back() + (geo[t].nsets + per_block - 1) / per_block);
        if (spw == 1) c->sa_blocks1 = sa_bs.back();  // a prefix: one set per wave only below kSaPairMinSets
        c->sa_max_blocks = std::max<int64_t>(c->sa_max_blocks, (geo[t].nsets + per_block - 1) / per_block);
    }
    c->nsa = (int32_t)sa_tab.size();
    c->sa_blocks = sa_bs.back();

    // clear the metadata (not the slot pool or staging), set "free" markers
    hipStream_t s0 = nullptr;
    for (int t = 0; t < T; ++t) {
        const Geom &ge = geo[t];
        HIP_TRY(hipMemsetAsync(ws + L.slot_row[t], 0xff, (size_t)ge.cap * 4, s0));
        HIP_TRY(hipMemsetAsync(ws + L.slot_score[t], 0, (size_t)ge.cap * 4, s0));
        HIP_TRY(hipMemsetAsync(ws + L.slot_flags[t], 0, (size_t)ge.cap * 4, s0));
        HIP_TRY(hipMemsetAsync(ws + L.slot_touch[t], 0xff, (size_t)ge.cap * 4, s0));
        HIP_TRY(hipMemsetAsync(ws + L.slot_cbit[t], 0, (size_t)ge.cap, s0));
        HIP_TRY(hipMemsetAsync(ws + L.map[t], 0xff, (size_t)ge.map_cap * 8, s0));
        HIP_TRY(hipMemsetAsync(ws + L.bitmap[t], 0, (size_t)ge.bm_words * 4, s0));
        HIP_TRY(hipMemsetAsync(ws + L.rank[t], 0xff, (size_t)ge.bm_words * 16, s0));  // stamp -1
        HIP_TRY(hipMemsetAsync(ws + L.seg[t], 0, (size_t)ge.nsets * 16, s0));
        if (cfg->policy == RECMG_LFU_BATCH) HIP_TRY(hipMemsetAsync(ws + L.freq[t], 0, (size_t)ge.rows * 4, s0));
        if (ge.ring_cap) {  // empty rings: no slot has an entry, no chunk a live one
            HIP_TRY(hipMemsetAsync(ws + L.slot_pos[t], 0xff, (size_t)ge.cap * 4, s0));
            HIP_TRY(hipMemsetAsync(ws + L.ring0[t], 0xff, (size_t)ge.ring_cap * 4, s0));
            HIP_TRY(hipMemsetAsync(ws + L.ring1[t], 0xff, (size_t)ge.ring_cap * 4, s0));
            HIP_TRY(hipMemsetAsync(ws + L.rcnt0[t], 0, (size_t)ge.ring_cap / kRingChunk * 4, s0));
            HIP_TRY(hipMemsetAsync(ws + L.rcnt1[t], 0, (size_t)ge.ring_cap / kRingChunk * 4, s0));
        }
    }
    HIP_TRY(hipMemsetAsync(ws + L.st, 0, sizeof(TState) * T, s0));
    HIP_TRY(hipMemsetAsync(ws + L.tstart, 0, 8 * (T + 1), s0));
    HIP_TRY(hipMemsetAsync(ws + L.pstart, 0, 8 * (T + 1), s0));
    HIP_TRY(hipMemsetAsync(ws + L.ftstart, 0, 8 * (T + 1), s0));
    HIP_TRY(hipMemsetAsync(ws + L.err, 0, 4, s0));
    HIP_TRY(hipMemsetAsync(ws + L.hist, 0, 4 * (size_t)kRadix * T, s0));
    HIP_TRY(hipMemcpy(ws + L.tabs, tabs.data(), sizeof(DTable) * T, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(ws + L.bm_block_start, bstart.data(), 4 * (T + 1), hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(ws + L.pool_btab, c->pool_order.data(), 4 * T, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(ws + L.sa_bstart, sa_bs.data(), 4 * sa_bs.size(), hipMemcpyHostToDevice));
    if (!sa_tab.empty()) HIP_TRY(hipMemcpy(ws + L.sa_btab, sa_tab.data(), 4 * sa_tab.size(), hipMemcpyHostToDevice));
    launch_init_state(g, c->max_cap, s0);
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipDeviceSynchronize());

    c->copy_stream = static_cast<hipStream_t>(cfg->copy_stream);
    for (hipEvent_t *e : {&c->ev_src, &c->ev_pool, &c->ev_fwd, &c->ev_plc, &c->ev_fill[0], &c->ev_fill[1]})
        HIP_TRY(hipEventCreateWithFlags(e, hipEventDisableTiming));
    if (c->has_staged) {
        char *hs = static_cast<char *>(cfg->host_staging);
        c->h_mrows = reinterpret_cast<int32_t *>(hs + L.h_mrows);
        c->h_rows = hs + L.h_rows;
        c->h_fsrc = reinterpret_cast<int32_t *>(hs + L.h_fsrc);
        c->h_frows = hs + L.h_frows;
        c->h_np = reinterpret_cast<int32_t *>(hs + L.h_np);
        c->he_st = reinterpret_cast<TState *>(hs + L.h_early);
        c->he_pstart = reinterpret_cast<int64_t *>(hs + L.h_early + sizeof(TState) * T);
        c->he_err = reinterpret_cast<int32_t *>(hs + L.h_early + sizeof(TState) * T + 8 * (T + 1));
        c->h_pstart.resize(T + 1);
        c->h_ftstart.resize(T + 1);
        HIP_TRY(hipEventCreateWithFlags(&c->ev_ready, hipEventDisableTiming));
        HIP_TRY(hipEventCreateWithFlags(&c->ev_copied, hipEventDisableTiming));
        HIP_TRY(hipEventCreateWithFlags(&c->ev_np, hipEventDisableTiming));
    }
    c->h_st.resize(T);
    c->h_tstart.resize(T + 1);
    *out = c.release();
    g_last_error.clear();
    return RECMG_OK;
}

}  // namespace

extern "C" {

int32_t recmg_apply_placement(recmg_cache_t *c, const int32_t *prefetch_rows, const int64_t *prefetch_offsets,
                              int64_t num_prefetch, const uint8_t *cache_bits, void *stream) {
    int32_t rc = check_handle(c);
    if (rc) return rc;
    if (!prefetch_offsets) return fail(RECMG_E_INVALID, "prefetch_offsets is NULL");
    if (num_prefetch < 0 || num_prefetch > c->cfg.max_prefetch)
        return fail(RECMG_E_INVALID, "num_prefetch out of [0, max_prefetch]");
    if (num_prefetch > 0 && !prefetch_rows) return fail(RECMG_E_INVALID, "prefetch_rows is NULL");
    if ((rc = set_device(c))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (c->cfg.validate && (rc = host_check_ids(prefetch_rows, prefetch_offsets, c->T + 1, 1, num_prefetch, c->geo, s)))
        return rc;
    const int64_t b = c->placements;
    if (b + 2 >= (int64_t(1) << 31)) return fail(RECMG_E_STATE, "placement count exhausted");
    EnqueueGuard guard(c);
    // what this placement reads from calls on other streams: the latest
    // forward's distinct rows, misses and sources; the latest placement's state
    if (c->fwd_ev && c->fwd_stream != s) HIP_TRY(hipStreamWaitEvent(s, c->ev_src, 0));
    if (c->plc_ev && c->plc_stream != s) HIP_TRY(hipStreamWaitEvent(s, c->ev_plc, 0));
    const int q = (int)(c->placements & 1);
    if (c->fill_rec[q]) HIP_TRY(hipStreamWaitEvent(s, c->ev_fill[q], 0));  // it read this parity's fill list
    // STAGED: the host rewrites its staging of fill sources and rows, which
    // the previous fill's copies may still read
    if (c->has_staged && c->fill_rec[q ^ 1]) HIP_TRY(hipStreamWaitEvent(s, c->ev_fill[q ^ 1], 0));
    c->g.staging = c->stage[c->cur];  // misses of the latest forward
    c->g.fill_src = c->fill_src_buf[q];
    c->g.fill_slot = c->fill_slot_buf[q];
    int64_t *fdesc = c->fdesc_buf[q];
    const DGlobal &g = c->g;
    PlcParams p{};
    p.prio = c->cfg.policy == RECMG_PRIORITY;
    p.lfu = c->cfg.policy == RECMG_LFU_BATCH;
    p.es = c->cfg.eviction_speed;
    p.lru_touch = (int32_t)b;
    p.pscore = p.prio ? p.es : p.lfu ? 0 : (int32_t)(b + 1);
    p.have_fwd = c->have_fwd ? 1 : 0;
    p.last_stamp = c->have_fwd ? (int32_t)(c->forwards - 1) : -2;
    p.rowbits = c->rowbits;
    // largest score a key can hold (an LFU count grows by at most one per placement)
    const int64_t maxscore = p.prio ? (int64_t)p.es + 1 : b + 1;
    p.total_bits = bitlen((uint64_t)maxscore) + p.rowbits;
    if (p.total_bits < 1) p.total_bits = 1;
    p.passes = (p.total_bits + kRadixBits - 1) / kRadixBits;

    {
        StageTimer tm(c, RECMG_STAGE_PLC_CLASSIFY, s);
        launch_plc_prep(g, prefetch_offsets, num_prefetch, p.have_fwd, s);
        if (p.prio && cache_bits && c->have_fwd) launch_plc_bits(g, cache_bits, c->last_n, s);
        if (p.lfu && c->have_fwd) launch_plc_freq(g, c->last_n, s);
        if (num_prefetch > 0) {
            launch_mark(g, prefetch_rows, g.pstart, num_prefetch, s);
            launch_dedup(g, EMIT_PREFETCH,
                         reinterpret_cast<int32_t *>(reinterpret_cast<char *>(g.st) + offsetof(TState, pcount)),
                         (int)(sizeof(TState) / 4), 0, c->max_nblk, s);
            launch_plc_classify(g, p.last_stamp, num_prefetch, s);
        }
    }
    // fully associative STAGED tables: their new prefetch candidates go to the
    // host now, so that it gathers their rows while the GPU ranks (early_gather)
    const bool early = c->has_staged_fa && num_prefetch > 0;
    if (early) {
        HIP_TRY(hipMemcpyAsync(c->he_st, g.st, sizeof(TState) * c->T, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(c->he_pstart, g.pstart, 8 * (c->T + 1), hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(c->h_np, g.NP, 4 * (size_t)num_prefetch, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipMemcpyAsync(c->he_err, g.err, 4, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipEventRecord(c->ev_np, s));
    }
    const int64_t cand = (c->have_fwd ? c->last_n : 0) + num_prefetch;
    const int64_t per_table = c->max_cap + (cand + c->T - 1) / c->T;
    const int64_t cand_grid = std::min<int64_t>(std::max<int64_t>(cand / c->T, 1024), cand + 1);
    // resident rings: a table's zones hold its pending rows (at most the last
    // placement's prefetch rows) and the last batch's distinct rows
    const int64_t ring_items = ((c->have_fwd ? c->last_n : 0) + c->plc_np_last + num_prefetch + c->T - 1) / c->T;
    if (c->has_fa) {
        StageTimer tm(c, RECMG_STAGE_PLC_RANK, s);
        if (c->has_scan_fa) launch_plc_rank(g, p, per_table, s);
        if (c->has_ring) launch_ring_rank(g, p, ring_items, s);
    }
    {
        StageTimer tm(c, RECMG_STAGE_PLC_APPLY, s);
        if (c->has_scan_fa) launch_plc_evict(g, p, c->max_cap, s);
        if (c->has_ring) launch_ring_evict(g, p, ring_items, c->max_ring_chunks, s);
        if (c->has_fa) launch_plc_admit(g, p, c->max_cap, c->max_map, cand_grid, s);
        if (c->has_ring) launch_ring_store(g, p, ring_items, c->max_cap, q, s);
        if (c->has_sa)
            launch_sa_place(g, p, c->have_fwd ? c->last_n : 0, num_prefetch, c->nsa, c->sa_blocks1, c->sa_blocks,
                            c->sa_max_blocks, s);
    }
    launch_plc_finalize(g, fdesc, c->cfg.stats_log_calls ? c->calls % c->cfg.stats_log_calls : -1, s);
    HIP_TRY(hipEventRecord(c->ev_plc, s));
    hipStream_t fs = c->copy_stream ? c->copy_stream : s;
    if (early) {
        // the host gathers while the kernels above run; the copies go on the
        // fill stream ahead of the fill (the last fill to read fstage has
        // ended: this placement's stream waited for it)
        StageTimer tm(c, RECMG_STAGE_PLC_FILL, fs);
        if ((rc = early_gather(c, fs))) return rc;
    }
    // The fill overwrites the slots of evicted rows: it waits for the latest
    // forward's pooled kernel, which may read them, and for this placement.
    // On the copy stream it overlaps the next forward's dedup and probe (and a
    // placement on a stream of its own overlaps the previous fill); that
    // forward's pooled kernel waits for it.
    if (fs != s) HIP_TRY(hipStreamWaitEvent(fs, c->ev_plc, 0));
    if (c->fwd_ev && c->fwd_stream != fs) HIP_TRY(hipStreamWaitEvent(fs, c->ev_pool, 0));
    // The previous placement's fill may still write slots this placement has
    // just freed and handed to other rows.  On one fill stream the two fills
    // run in order; on different ones (no copy stream, placements on
    // different streams) this fill waits for it, and so does every forward
    // that waits for this fill.
    if (c->fill_rec[q ^ 1] && c->fill_stream[q ^ 1] != fs) HIP_TRY(hipStreamWaitEvent(fs, c->ev_fill[q ^ 1], 0));
    {
        StageTimer tm(c, RECMG_STAGE_PLC_FILL, fs);
        // Zero-copy tables' rows are read from the host by the kernel, at
        // once (beside the host gather of the STAGED tables' rows); STAGED
        // tables' rows once the host has staged them.
        DispatchTimer dt(c, RECMG_STAGE_PLC_FILL, true);
        if (c->has_zc) launch_plc_fill(g, fdesc, FILL_ZERO_COPY, fs, dt.a, c->has_staged ? nullptr : dt.b);
        if (c->has_staged) {
            if (c->has_staged_sa && (rc = staged_fill(c, s, fs))) return rc;  // host-staged rows
            launch_plc_fill(g, fdesc, FILL_STAGED, fs, c->has_zc ? nullptr : dt.a, dt.b);
        }
        dt.issued();
    }
    HIP_TRY(hipEventRecord(c->ev_fill[q], fs));
    c->fill_rec[q] = true;
    c->fill_stream[q] = fs;
    c->fill_last = q;
    HIP_TRY(hipGetLastError());
    guard.done = true;
    c->placements++;
    c->calls++;
    c->plc_np = num_prefetch;
    c->plc_np_last = num_prefetch;
    c->have_fwd = false;
    c->last_stream = s;
    c->plc_stream = s;
    c->plc_ev = true;
    return RECMG_OK;
}

int32_t recmg_embbag_forward(recmg_cache_t *c, const int32_t *indices, const int64_t *offsets, int64_t num_indices,
                             int32_t bags_per_table, float *out, void *stream) {
    int32_t rc = check_handle(c);
    if (rc) return rc;
    const int64_t B = bags_per_table, n = num_indices;
    if (B < 0 || B > c->cfg.max_bags_per_table) return fail(RECMG_E_INVALID, "bags_per_table out of [0, max]");
    if (n < 0 || n > c->cfg.max_indices) return fail(RECMG_E_INVALID, "num_indices out of [0, max_indices]");
    if (!offsets) return fail(RECMG_E_INVALID, "offsets is NULL");
    if (n > 0 && !indices) return fail(RECMG_E_INVALID, "indices is NULL");
    if (B > 0 && !out) return fail(RECMG_E_INVALID, "out is NULL");
    if ((rc = set_device(c))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (c->cfg.validate && (rc = host_check_ids(indices, offsets, (int64_t)c->T * B + 1, B, n, c->geo, s))) return rc;
    if (c->forwards + 1 >= (int64_t(1) << 31)) return fail(RECMG_E_STATE, "forward count exhausted");
    EnqueueGuard guard(c);
    // what this forward needs from calls on other streams: the latest
    // placement's state (its fill is waited for before the pooled kernel) and
    // the end of the latest forward, whose per-index arrays this one rewrites
    if (c->plc_ev && c->plc_stream != s) HIP_TRY(hipStreamWaitEvent(s, c->ev_plc, 0));
    if (c->fwd_ev && c->fwd_stream != s) HIP_TRY(hipStreamWaitEvent(s, c->ev_fwd, 0));
    const DGlobal &g = c->g;
    if (c->pool_B != (int32_t)B) {
        // blocks of the pooled kernels: tables grouped by kernel kind, one
        // launch per kind over its contiguous range of blocks
        c->pool_bstart.assign(c->T + 1, 0);
        c->pool_launches.clear();
        for (int k = 0; k < c->T; ++k) {
            const Geom &ge = c->geo[c->pool_order[k]];
            const int32_t nb = (int32_t)((B + ge.bpb - 1) / ge.bpb);
            c->pool_bstart[k + 1] = c->pool_bstart[k] + nb;
            if (c->pool_launches.empty() || c->pool_launches.back().kind != ge.kind)
                c->pool_launches.push_back({ge.kind, c->pool_bstart[k], 0, k, nb});
            PoolLaunch &pl = c->pool_launches.back();
            pl.nblk += nb;
            if (pl.nbt != nb) pl.nbt = 0;  // blocks per table differ: the kernel searches bstart
        }
        HIP_TRY(hipMemcpyAsync(static_cast<char *>(c->cfg.device_workspace) + c->L.pool_bstart, c->pool_bstart.data(),
                               4 * (c->T + 1), hipMemcpyHostToDevice, s));
        HIP_TRY(hipStreamSynchronize(s));
        c->pool_B = (int32_t)B;
        c->pool_blocks = c->pool_bstart[c->T];
    }
    const int32_t stamp = (int32_t)c->forwards;
    c->cur ^= 1;  // the other staging buffer: a pending fill may still read this one
    c->g.staging = c->stage[c->cur];
    {
        StageTimer tm(c, RECMG_STAGE_FWD_DEDUP, s);
        launch_fwd_prep(g, offsets, (int32_t)B, n, s);
        if (n > 0) {
            launch_mark(g, indices, g.tstart, n, s);
            launch_dedup(g, EMIT_FORWARD,
                         reinterpret_cast<int32_t *>(reinterpret_cast<char *>(g.st) + offsetof(TState, ucount)),
                         (int)(sizeof(TState) / 4), stamp, c->max_nblk, s);
            launch_fwd_probe(g, stamp, n, s);
            launch_fwd_src(g, indices, n, s);
            if (c->plc_np >= 0) launch_fwd_cover(g, stamp, c->plc_np, s);
        }
    }
    HIP_TRY(hipEventRecord(c->ev_src, s));  // a placement on another stream may start here
    if (n > 0) {
        StageTimer tm(c, RECMG_STAGE_FWD_FETCH, s);
        if (!c->has_staged) {
            DispatchTimer dt(c, RECMG_STAGE_FWD_FETCH, true);
            launch_fetch(g, s, dt.a, dt.b);
            dt.issued();
        } else if ((rc = staged_fetch(c, s))) {  // launches the zero-copy tables' fetch too
            return rc;
        }
    }
    if (c->fill_last >= 0) {  // rows the latest placement admitted
        HIP_TRY(hipStreamWaitEvent(s, c->ev_fill[c->fill_last], 0));
        c->fill_last = -1;
    }
    {
        // the pooled kernel is timed by events its own dispatch records
        hipEvent_t a = nullptr, b = nullptr;
        if (c->timing >= 1 && c->pool_blocks > 0) {
            a = take_event(c);
            b = a ? take_event(c) : nullptr;
            if (!b && a) {
                c->ev_free.push_back(a);
                a = nullptr;
            }
        }
        char *ws = static_cast<char *>(c->cfg.device_workspace);
        launch_pool(g, offsets, (int32_t)B, out, reinterpret_cast<const int32_t *>(ws + c->L.pool_bstart),
                    reinterpret_cast<const int32_t *>(ws + c->L.pool_btab), c->T, c->pool_launches.data(),
                    (int)c->pool_launches.size(), a, b, s);
        if (a) c->marks.push_back({RECMG_STAGE_FWD_POOL, a, b});
    }
    HIP_TRY(hipEventRecord(c->ev_pool, s));  // the next fill may overwrite slots from here on
    launch_fwd_finalize(g, c->cfg.stats_log_calls ? c->calls % c->cfg.stats_log_calls : -1, s);
    HIP_TRY(hipEventRecord(c->ev_fwd, s));
    HIP_TRY(hipGetLastError());
    guard.done = true;
    c->forwards++;
    c->calls++;
    c->plc_np = -1;  // coverage counts against the placement just before a forward only
    c->have_fwd = true;
    c->last_n = n;
    c->last_stream = s;
    c->fwd_stream = s;
    c->fwd_ev = true;
    return RECMG_OK;
}

static_assert(sizeof(recmg_table_stats_t) == 8 * (kNumStats + 1), "counter layout of recmg_table_stats_t");

int32_t recmg_stats(recmg_cache_t *c, recmg_table_stats_t *last, recmg_table_stats_t *total, int32_t *resident_dump,
                    int64_t dump_capacity, int64_t *resident_counts) {
    int32_t rc = check_handle(c);
    if (rc) return rc;
    if ((rc = set_device(c))) return rc;
    hipStream_t s = c->last_stream;
    HIP_TRY(sync_all(c));
    const int T = c->T;
    std::vector<TState> st(T);
    int32_t err = 0;
    HIP_TRY(hipMemcpy(st.data(), c->g.st, sizeof(TState) * T, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(&err, c->g.err, 4, hipMemcpyDeviceToHost));
    for (int t = 0; t < T; ++t) {
        for (int which = 0; which < 2; ++which) {
            recmg_table_stats_t *o = which == 0 ? last : total;
            if (!o) continue;
            const int64_t *v = which == 0 ? st[t].last : st[t].total;
            int64_t *dst = &o[t].lookups;
            for (int k = 0; k < kNumStats; ++k) dst[k] = v[k];
            o[t].digest = st[t].digest;
        }
    }
    if (err & ERR_INTERNAL) return fail(RECMG_E_STATE, "device error flag: slot accounting invariant failed");
    if (err) return fail(RECMG_E_RANGE, "device error flag set (row id out of range or malformed offsets)");
    if (resident_dump || resident_counts) {
        int64_t need = 0;
        for (int t = 0; t < T; ++t) need += st[t].n_res;
        if (resident_dump && dump_capacity < need) return fail(RECMG_E_INVALID, "dump_capacity too small");
        launch_mark_resident(c->g, c->max_cap, s);
        launch_dedup(c->g, EMIT_DUMP, c->g.dump_count, 1, 0, c->max_nblk, s);
        HIP_TRY(hipGetLastError());
        std::vector<int32_t> cnt(T);
        HIP_TRY(hipMemcpyAsync(cnt.data(), c->g.dump_count, 4 * T, hipMemcpyDeviceToHost, s));
        HIP_TRY(hipStreamSynchronize(s));
        int64_t at = 0, coff = 0;
        for (int t = 0; t < T; ++t) {
            if (resident_counts) resident_counts[t] = cnt[t];
            if (resident_dump && cnt[t])
                HIP_TRY(hipMemcpy(resident_dump + at, c->g.dump + coff, 4 * (size_t)cnt[t], hipMemcpyDeviceToHost));
            at += cnt[t];
            coff += c->geo[t].cap;
        }
    }
    g_last_error.clear();
    return RECMG_OK;
}

int32_t recmg_stats_log(recmg_cache_t *c, recmg_table_stats_t *out, int64_t first_call, int64_t n_calls,
                        int64_t *calls_made) {
    int32_t rc = check_handle(c);
    if (rc) return rc;
    if (calls_made) *calls_made = c->calls;
    if (n_calls == 0) return RECMG_OK;
    const int64_t cap = c->cfg.stats_log_calls;
    if (!out || n_calls < 0 || first_call < 0 || first_call + n_calls > c->calls || first_call < c->calls - cap)
        return fail(RECMG_E_INVALID, "calls outside the stats log (the latest stats_log_calls calls are kept)");
    if ((rc = set_device(c))) return rc;
    HIP_TRY(sync_all(c));
    const size_t rec = sizeof(recmg_table_stats_t) * (size_t)c->T;
    for (int64_t k = first_call; k < first_call + n_calls; ++k)
        HIP_TRY(hipMemcpy(reinterpret_cast<char *>(out) + (k - first_call) * rec,
                          reinterpret_cast<const char *>(c->g.stat_log) + (k % cap) * rec, rec, hipMemcpyDeviceToHost));
    int32_t err = 0;
    HIP_TRY(hipMemcpy(&err, c->g.err, 4, hipMemcpyDeviceToHost));
    if (err) return fail(RECMG_E_RANGE, "device error flag set (row id out of range or malformed offsets)");
    g_last_error.clear();
    return RECMG_OK;
}

int32_t recmg_set_timing(recmg_cache_t *c, int32_t level) {
    int32_t rc = check_handle(c);
    if (rc) return rc;
    if (level < 0 || level > 2) return fail(RECMG_E_INVALID, "timing level must be 0, 1 or 2");
    c->timing = level;
    return RECMG_OK;
}

int32_t recmg_stage_times(recmg_cache_t *c, double *ms, int64_t *calls, int32_t reset) {
    int32_t rc = check_handle(c);
    if (rc) return rc;
    if (!ms) return fail(RECMG_E_INVALID, "ms is NULL");
    if ((rc = set_device(c))) return rc;
    // every interval on one time line (offsets from the first mark's start)
    std::vector<std::pair<double, double>> link;
    for (auto &m : c->marks) {
        HIP_TRY(hipEventSynchronize(m.b));
        float t = 0.f, t0 = 0.f, t1 = 0.f;
        HIP_TRY(hipEventElapsedTime(&t, m.a, m.b));
        c->stage_ms[m.stage] += t;
        c->stage_calls[m.stage] += 1;
        if (m.stage == RECMG_STAGE_FWD_FETCH || m.stage == RECMG_STAGE_PLC_FILL) {
            HIP_TRY(hipEventElapsedTime(&t0, c->marks[0].a, m.a));
            HIP_TRY(hipEventElapsedTime(&t1, c->marks[0].a, m.b));
            link.emplace_back(t0, t1);
        }
    }
    std::sort(link.begin(), link.end());
    double busy = 0, cur_a = 0, cur_b = -1;
    for (auto &iv : link) {
        if (iv.first > cur_b) {
            if (cur_b > cur_a) busy += cur_b - cur_a;
            cur_a = iv.first;
            cur_b = iv.second;
        } else if (iv.second > cur_b) {
            cur_b = iv.second;
        }
    }
    if (cur_b > cur_a) busy += cur_b - cur_a;
    c->stage_ms[RECMG_STAGE_HOST_LINK] += busy;
    c->stage_calls[RECMG_STAGE_HOST_LINK] += (int64_t)link.size();
    for (auto &m : c->marks) {
        c->ev_free.push_back(m.a);
        c->ev_free.push_back(m.b);
    }
    c->marks.clear();
    for (int k = 0; k < RECMG_NUM_STAGES; ++k) {
        ms[k] = c->stage_ms[k];
        if (calls) calls[k] = c->stage_calls[k];
        if (reset) {
            c->stage_ms[k] = 0;
            c->stage_calls[k] = 0;
        }
    }
    return RECMG_OK;
}

int32_t recmg_cache_destroy(recmg_cache_t *c) {
    if (!c) return RECMG_OK;
    if (c->magic != kMagic) return fail(RECMG_E_STATE, "handle is not live");
    (void)set_device(c);
    int32_t rc = RECMG_OK;
    if (sync_all(c) != hipSuccess) rc = fail(RECMG_E_HIP, "synchronize failed at destroy");
    c->magic = 0;
    if (c->static_ws) {
        std::lock_guard<std::mutex> lock(g_static_mu);
        if (g_static_owner[c->device] == c) g_static_owner[c->device] = nullptr;
    }
    delete c;  // destroys the handle's events
    return rc;
}

}  // extern "C"
