/*
 * CPU oracle for the tiered pooled-embedding lookup and its cache-state machine
 * (RecMG, "Machine Learning-Guided Memory Optimization for DLRM Inference on
 * Tiered Memory", HPCA'25, arXiv 2511.08568).
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the package's smoke check and the
 * benchmark's CPU-baseline leg load the library built from this file.  The HIP
 * path never calls it; the two share no source, header, helper or table.
 *
 * Plain and slow on purpose.  Every set of the definition is a byte array
 * indexed by row id; placement sorts the whole candidate set by key; pooled
 * sums are accumulated in double and rounded once to float.
 *
 * What it computes, per table t (caches are partitioned per table; fully
 * associative unless `ways` > 0, see the set-associative placement below):
 *
 * Forward on one batch (Sec. II, pooling by summation; Sec. VII-E for the
 * three-way split of accesses into cache hits, prefetch hits and on-demand
 * fetches):
 *   U = distinct rows of the batch, H = U ∩ R, M = U \ R.
 *   lookups, unique = |U|, hits = |H|, hits_prefetch = |{r in H : pf(r)}|,
 *   misses = |M| (on-demand fetches), ondemand_bytes = |M| * row_bytes.
 *   prefetch_covered = |set(P) ∩ U| with P the prefetch list of the placement
 *   just before this forward (0 if another forward came between): the
 *   numerator of Sec. IV's coverage (Eq. coverage), whose denominator is |U|.
 *   out[bag] = sum of the bag's rows, repeats counted, empty bag = 0.
 *   The forward reads residency and never changes it.
 *
 * Placement before the next batch (Sec. VI-B: load_embeddings, Alg. 1, and
 * gpu_buffer_populate, Alg. 2, run at the end of each batch; eviction_speed ES
 * defaults to 4).  It consumes U and M of the most recent forward, the caching
 * bit of every access of that forward and the prefetch list P:
 *   1. PRIORITY: every resident row ages once, s <- max(0, s - 1) (Alg. 2's
 *      saturating decrement, applied once per placement).
 *   2. rows of U that are resident lose their prefetch flag.
 *   3. touch: for r in U, s(r) <- b-1 under LRU_BATCH (b = index of this
 *      placement, so b-1 is the batch just run), or c(r) + ES under PRIORITY
 *      (Alg. 1's priority = C + eviction_speed), with c(r) the OR of r's bits,
 *      or f(r) under LFU_BATCH, f(r) being the number of batches that have
 *      accessed r so far (counted for every row, resident or not, by the
 *      placement that consumes the batch; the 32-way LFU baseline of
 *      Sec. VII-B at batch granularity).
 *   4. prefetch: for r in set(P), s(r) <- max(s(r) if r in R or M, else -inf,
 *      b under LRU_BATCH or ES under PRIORITY) (Alg. 1's prefetch priority);
 *      under LFU_BATCH a prefetched row keeps its frequency f(r).
 *   5. K = R ∪ M ∪ set(P); R' = the min(Cap, |K|) members with the largest
 *      key (s(r), r): the lowest score is evicted first, and among equal
 *      scores the lower row id goes first (Alg. 2's minimum-priority victim).
 *   6. newly admitted rows get pf(r) = [r in P].
 *   Counters: evicted, admitted_miss, prefetch_fill, prefetch_resident,
 *   prefetch_dropped, miss_dropped, resident, prefetch_bytes,
 *   prefetch_distinct = |set(P)|, and the digest
 *   sum over R' of SplitMix64's output mix of ((t << 40) | r), mod 2^64.
 *
 * Set-associative placement (ways W > 0; Sec. VI-B: the buffer is TorchRec's
 * software cache, whose production form is W-way set-associative, Sec. VII-B
 * and VII-E).  Per table, S = floor(Cap / W) sets of W ways; row r belongs to
 * set r mod S (no sets when S = 0: nothing is ever resident).  Alg. 1 and
 * Alg. 2 run literally inside each set, one event at a time:
 *   A. rows of U that are resident lose their prefetch flag and take the touch
 *      score (as in step 3 above; no aging here);
 *   B. every miss of M, in ascending row order, is inserted with its touch
 *      score;
 *   C. every row of set(P), in ascending row order: if resident, its score
 *      becomes max(score, b or ES); otherwise it is inserted with score b
 *      (LRU_BATCH) or ES (PRIORITY).
 *   insert(r, v) in r's set: the lowest free way if there is one; otherwise
 *   Alg. 2 on the set: the victim is the lowest way holding the minimum score
 *   (scores before this scan's aging), then, under PRIORITY only, every way
 *   of the set ages by one, saturating at 0; r takes the victim's way.
 *   A row whose way at the end differs from its way at the start (newly
 *   admitted, or evicted and brought back into another way) gets
 *   pf(r) = [r in P]; other residents keep their flag.  Counters are those of
 *   the fully associative form, except that prefetch_fill counts every row
 *   read from the host: rows of (R' \ R) \ M and rows of R ∩ R' that moved.
 *
 * Compile-time ORACLE_MUTANT = k (k > 0) plants one known mistake; the test
 * suite builds those variants on the CPU to show that its pins catch them.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef ORACLE_MUTANT
#define ORACLE_MUTANT 0
#endif

enum { O_F32 = 0, O_F16 = 1, O_BF16 = 2 };
enum { O_LRU_BATCH = 0, O_PRIORITY = 1, O_LFU_BATCH = 2 };
enum { O_OK = 0, O_E_RANGE = -1, O_E_INVALID = -2 };

typedef struct {
    int64_t n, cap;
    int32_t d, dtype, row_bytes;
    const void *vals;
    /* cache state: resident set, score and prefetch flag, indexed by row */
    uint8_t *in_r, *pf;
    int64_t *s;
    int32_t *res; /* resident rows, unordered */
    int64_t nres;
    /* what the last forward leaves for the next placement */
    int have_fwd;
    int32_t *last_idx;
    int64_t nlast, last_base; /* this table's slice of the last batch */
    int32_t *U, *M;
    int64_t nU, nM;
    /* scratch marks, indexed by row; all zero between calls */
    uint8_t *in_u, *in_m, *in_p, *c;
    /* the distinct prefetch rows of the latest placement, for the next
     * forward's coverage (Sec. IV, Eq. coverage); have_plc: no forward since */
    int32_t *lastP;
    int64_t nlastP;
    int have_plc;
    /* counters */
    int64_t fwd[7];
    int64_t plc[9];
    uint64_t digest;
    /* LFU_BATCH: number of batches that accessed each row (kept for every row) */
    int64_t *freq;
    /* set-associative form: nsets sets of `ways` rows each (-1 = free way) */
    int64_t nsets;
    int32_t *way_row, *way_row0;
    uint8_t *in_r0;
} otab;

typedef struct {
    int32_t T, policy, es, nthreads, ways;
    int64_t placements, forwards;
    otab *t;
} oracle_t;

/* SplitMix64 output mix (Steele, Lea & Flood, OOPSLA 2014). */
uint64_t oracle_splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* IEEE 754 binary16 -> double, from the format's definition. */
static double half_to_double(uint16_t h) {
    int sign = h >> 15, e = (h >> 10) & 31, m = h & 1023;
    double v;
    if (e == 0) v = ldexp((double)m, -24);
    else if (e == 31) v = m ? NAN : INFINITY;
    else v = ldexp((double)(1024 + m), e - 25);
    return sign ? -v : v;
}

/* bfloat16 -> double: the upper half of a binary32. */
static double bf16_to_double(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static double elem(const otab *tb, int64_t row, int32_t k) {
    int64_t i = row * tb->d + k;
    switch (tb->dtype) {
    case O_F32: return (double)((const float *)tb->vals)[i];
    case O_F16: return half_to_double(((const uint16_t *)tb->vals)[i]);
    default: return bf16_to_double(((const uint16_t *)tb->vals)[i]);
    }
}

void oracle_destroy(void *h) {
    oracle_t *o = (oracle_t *)h;
    if (!o) return;
    for (int32_t t = 0; t < o->T; ++t) {
        otab *tb = &o->t[t];
        free(tb->in_r); free(tb->pf); free(tb->s); free(tb->res);
        free(tb->last_idx); free(tb->U); free(tb->M);
        free(tb->in_u); free(tb->in_m); free(tb->in_p); free(tb->c);
        free(tb->lastP);
        free(tb->way_row); free(tb->way_row0); free(tb->in_r0); free(tb->freq);
    }
    free(o->t);
    free(o);
}

void *oracle_create(int32_t T, const int64_t *rows, const int32_t *dims, const int32_t *dtypes,
                    const void *const *tables, const int64_t *caps, int32_t policy, int32_t es,
                    int32_t nthreads, int32_t ways) {
    if (T <= 0 || !rows || !dims || !dtypes || !tables || !caps) return NULL;
    if (policy != O_LRU_BATCH && policy != O_PRIORITY && policy != O_LFU_BATCH) return NULL;
    if (ways < 0) return NULL;
    oracle_t *o = (oracle_t *)calloc(1, sizeof(oracle_t));
    o->T = T; o->policy = policy; o->es = es; o->nthreads = nthreads > 0 ? nthreads : 1; o->ways = ways;
    o->t = (otab *)calloc((size_t)T, sizeof(otab));
    for (int32_t t = 0; t < T; ++t) {
        otab *tb = &o->t[t];
        if (rows[t] <= 0 || dims[t] <= 0 || caps[t] < 0 || dtypes[t] < 0 || dtypes[t] > 2 || !tables[t]) {
            oracle_destroy(o);
            return NULL;
        }
        tb->n = rows[t]; tb->d = dims[t]; tb->dtype = dtypes[t]; tb->vals = tables[t];
        tb->cap = caps[t] < rows[t] ? caps[t] : rows[t];
        tb->row_bytes = dims[t] * (dtypes[t] == O_F32 ? 4 : 2);
        size_t n = (size_t)tb->n;
        tb->in_r = (uint8_t *)calloc(n, 1); tb->pf = (uint8_t *)calloc(n, 1);
        tb->s = (int64_t *)calloc(n, sizeof(int64_t));
        tb->res = (int32_t *)malloc(sizeof(int32_t) * (size_t)(tb->cap + 1));
        tb->in_u = (uint8_t *)calloc(n, 1); tb->in_m = (uint8_t *)calloc(n, 1);
        tb->in_p = (uint8_t *)calloc(n, 1); tb->c = (uint8_t *)calloc(n, 1);
        if (policy == O_LFU_BATCH) tb->freq = (int64_t *)calloc(n, sizeof(int64_t));
        if (ways > 0) {
            tb->nsets = tb->cap / ways;
            size_t nw = (size_t)(tb->nsets * ways) + 1;
            tb->way_row = (int32_t *)malloc(sizeof(int32_t) * nw);
            tb->way_row0 = (int32_t *)malloc(sizeof(int32_t) * nw);
            for (size_t k = 0; k < nw; ++k) tb->way_row[k] = -1;
            tb->in_r0 = (uint8_t *)calloc(n, 1);
        }
    }
    return o;
}

/* ---------------------------------------------------------------- placement */

typedef struct { int64_t s; int32_t r; } okey;

/* Descending by (score, row): the largest keys come first and are kept. */
static int key_desc(const void *a, const void *b) {
    const okey *x = (const okey *)a, *y = (const okey *)b;
    if (x->s != y->s) return x->s > y->s ? -1 : 1;
#if ORACLE_MUTANT == 1 /* planted: among equal scores the higher id is evicted first */
    if (x->r != y->r) return x->r < y->r ? -1 : 1;
#else
    if (x->r != y->r) return x->r > y->r ? -1 : 1;
#endif
    return 0;
}

static void place_table_sa(oracle_t *o, int32_t t, const int32_t *P, int64_t nP);

/* Score of a row the last batch touched, in placement b. */
static int64_t touch_score(const oracle_t *o, const otab *tb, int32_t r, int64_t b) {
    if (o->policy == O_LRU_BATCH) return b - 1;
    if (o->policy == O_PRIORITY) return (int64_t)tb->c[r] + o->es;
    return tb->freq[r];
}

/* Score a prefetch gives a row not resident and not missed (the prefetch
 * score); a resident or missed row keeps the larger of its score and this.
 * LFU_BATCH ranks a prefetched row by its frequency and gives no floor. */
static int64_t prefetch_score(const oracle_t *o, const otab *tb, int32_t r, int64_t b) {
    if (o->policy == O_LRU_BATCH) {
#if ORACLE_MUTANT == 7 /* planted: prefetch scored like a touch */
        return b - 1;
#else
        return b;
#endif
    }
    if (o->policy == O_PRIORITY) return o->es;
    return tb->freq[r];
}

static int64_t prefetch_floor(const oracle_t *o, const otab *tb, int32_t r, int64_t b) {
    return o->policy == O_LFU_BATCH ? 0 : prefetch_score(o, tb, r, b);
}

static void place_table(oracle_t *o, int32_t t, const int32_t *P, int64_t nP, const uint8_t *bits) {
    otab *tb = &o->t[t];
    const int64_t b = o->placements;
    const int prio = o->policy == O_PRIORITY;
    int64_t nU = tb->have_fwd ? tb->nU : 0, nM = tb->have_fwd ? tb->nM : 0;

    /* LFU_BATCH: one more batch for every row the last batch accessed */
    if (o->policy == O_LFU_BATCH && tb->have_fwd) {
#if ORACLE_MUTANT == 17 /* planted: frequency counts every access, not every batch */
        for (int64_t i = 0; i < tb->nlast; ++i) tb->freq[tb->last_idx[i]] += 1;
#else
        for (int64_t k = 0; k < nU; ++k) tb->freq[tb->U[k]] += 1;
#endif
    }
    /* c(r): OR of the caching bits over r's accesses in the last batch. */
    if (prio && bits && tb->have_fwd) {
        for (int64_t i = 0; i < tb->nlast; ++i) {
#if ORACLE_MUTANT == 4 /* planted: the last access's bit wins */
            tb->c[tb->last_idx[i]] = bits[tb->last_base + i] != 0;
#else
            if (bits[tb->last_base + i]) tb->c[tb->last_idx[i]] = 1;
#endif
        }
    }
    if (o->ways > 0) {
        place_table_sa(o, t, P, nP);
        return;
    }
    /* 1. aging (PRIORITY) */
#if ORACLE_MUTANT != 2 /* planted (2): no aging */
    if (prio)
        for (int64_t k = 0; k < tb->nres; ++k) {
            int32_t r = tb->res[k];
#if ORACLE_MUTANT == 9 /* planted: the decrement does not saturate at 0 */
            tb->s[r] = tb->s[r] - 1;
#else
            tb->s[r] = tb->s[r] > 0 ? tb->s[r] - 1 : 0;
#endif
        }
#endif
    /* 2. accessed residents lose their prefetch flag; 3. touch */
    for (int64_t k = 0; k < nU; ++k) {
        int32_t r = tb->U[k];
#if ORACLE_MUTANT != 6 /* planted (6): prefetch flag survives an access */
        if (tb->in_r[r]) tb->pf[r] = 0;
#endif
        tb->s[r] = touch_score(o, tb, r, b);
    }
    /* 4. prefetch scores over set(P) */
    int64_t np_new = 0, p_res = 0;
    int32_t *pnew = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nP + 1));
    free(tb->lastP);
    tb->lastP = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nP + 1));
    tb->nlastP = 0;
    for (int64_t k = 0; k < nP; ++k) {
        int32_t r = P[k];
        if (tb->in_p[r]) continue;
        tb->in_p[r] = 1;
        tb->lastP[tb->nlastP++] = r;
        if (tb->in_r[r] || tb->in_m[r]) {
#if ORACLE_MUTANT == 3 /* planted: prefetch overwrites the score */
            tb->s[r] = prefetch_floor(o, tb, r, b);
#else
            if (prefetch_floor(o, tb, r, b) > tb->s[r]) tb->s[r] = prefetch_floor(o, tb, r, b);
#endif
            if (tb->in_r[r]) ++p_res;
        } else {
            tb->s[r] = prefetch_score(o, tb, r, b);
            pnew[np_new++] = r;
        }
    }
    /* 5. K = R ∪ M ∪ set(P); keep the min(Cap, |K|) largest keys */
    int64_t nK = tb->nres + nM + np_new;
    okey *K = (okey *)malloc(sizeof(okey) * (size_t)(nK + 1));
    int64_t q = 0;
    for (int64_t k = 0; k < tb->nres; ++k) K[q].r = tb->res[k], K[q].s = tb->s[tb->res[k]], ++q;
    for (int64_t k = 0; k < nM; ++k) K[q].r = tb->M[k], K[q].s = tb->s[tb->M[k]], ++q;
    for (int64_t k = 0; k < np_new; ++k) K[q].r = pnew[k], K[q].s = tb->s[pnew[k]], ++q;
    qsort(K, (size_t)nK, sizeof(okey), key_desc);
    int64_t keep = nK < tb->cap ? nK : tb->cap;

    /* 6. apply; count */
    int64_t evicted = 0, adm_miss = 0, fill = 0, p_drop = 0, m_drop = 0;
    uint8_t *keepm = tb->in_u; /* all zero between calls; marks R' here */
    for (int64_t k = 0; k < keep; ++k) keepm[K[k].r] = 1;
    for (int64_t k = 0; k < tb->nres; ++k)
        if (!keepm[tb->res[k]]) { ++evicted; tb->in_r[tb->res[k]] = 0; tb->pf[tb->res[k]] = 0; }
    for (int64_t k = 0; k < nM; ++k) if (!keepm[tb->M[k]]) ++m_drop;
    for (int64_t k = 0; k < np_new; ++k) if (!keepm[pnew[k]]) ++p_drop;
    for (int64_t k = 0; k < nM; ++k)
        if (tb->in_p[tb->M[k]] && !keepm[tb->M[k]]) ++p_drop;
    uint64_t dig = 0;
    tb->nres = 0;
    for (int64_t k = 0; k < keep; ++k) {
        int32_t r = K[k].r;
        if (!tb->in_r[r]) {
            if (tb->in_m[r]) ++adm_miss; else ++fill;
            tb->in_r[r] = 1;
            /* every admitted row that P names is flagged, a miss of the last
               batch included (R16) */
#if ORACLE_MUTANT == 18 /* planted: an admitted miss that P names is not flagged */
            tb->pf[r] = tb->in_p[r] && !tb->in_m[r];
#else
            tb->pf[r] = tb->in_p[r];
#endif
        }
        tb->res[tb->nres++] = r;
#if ORACLE_MUTANT == 8 /* planted: digest forgets the table id */
        dig += oracle_splitmix64_mix((uint64_t)r);
#else
        dig += oracle_splitmix64_mix(((uint64_t)t << 40) | (uint64_t)r);
#endif
    }
    /* clear scratch marks */
    for (int64_t k = 0; k < keep; ++k) keepm[K[k].r] = 0;
    for (int64_t k = 0; k < nP; ++k) tb->in_p[P[k]] = 0;
    for (int64_t k = 0; k < nU; ++k) { tb->in_m[tb->U[k]] = 0; tb->c[tb->U[k]] = 0; }

    tb->plc[0] = evicted; tb->plc[1] = adm_miss; tb->plc[2] = fill; tb->plc[3] = p_res;
    tb->plc[4] = p_drop; tb->plc[5] = m_drop; tb->plc[6] = tb->nres; tb->plc[7] = fill * tb->row_bytes;
    tb->plc[8] = tb->nlastP;
    tb->digest = dig;
    tb->have_fwd = 0;
    tb->have_plc = 1;
    free(K);
    free(pnew);
}

/* --------------------------------------------------- set-associative placement */

static int cmp_row(const void *a, const void *b) {
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
#if ORACLE_MUTANT == 14 /* planted: events of a set taken in descending row order */
    return (x < y) - (x > y);
#else
    return (x > y) - (x < y);
#endif
}

static int64_t set_of(const otab *tb, int32_t r, int32_t ways) {
#if ORACLE_MUTANT == 16 /* planted: the set index taken modulo the ways */
    return ((int64_t)r % ways) % tb->nsets;
#else
    (void)ways;
    return (int64_t)r % tb->nsets;
#endif
}

/* Put row r with score v into its set (Alg. 1's fetch; Alg. 2 when the set is full). */
static void sa_insert(oracle_t *o, otab *tb, int32_t r, int64_t v) {
    const int32_t W = o->ways;
    if (tb->nsets == 0) return; /* no sets: r is dropped */
    int32_t *set = tb->way_row + set_of(tb, r, W) * W;
    int32_t w = -1;
    for (int32_t k = 0; k < W && w < 0; ++k)
        if (set[k] < 0) w = k;
    if (w < 0) {
        /* Alg. 2: scan the set for the lowest score; a later way replaces the
         * incumbent only if strictly lower */
#if ORACLE_MUTANT == 12 /* planted: the set ages before the victim is chosen */
        if (o->policy == O_PRIORITY)
            for (int32_t k = 0; k < W; ++k) tb->s[set[k]] = tb->s[set[k]] > 0 ? tb->s[set[k]] - 1 : 0;
#endif
        w = 0;
        for (int32_t k = 1; k < W; ++k)
#if ORACLE_MUTANT == 11 /* planted: among equal scores the last way is the victim */
            if (tb->s[set[k]] <= tb->s[set[w]]) w = k;
#else
            if (tb->s[set[k]] < tb->s[set[w]]) w = k;
#endif
#if ORACLE_MUTANT != 12 && ORACLE_MUTANT != 15
        if (o->policy == O_PRIORITY)
            for (int32_t k = 0; k < W; ++k) tb->s[set[k]] = tb->s[set[k]] > 0 ? tb->s[set[k]] - 1 : 0;
#endif
        tb->in_r[set[w]] = 0;
    }
    set[w] = r;
    tb->in_r[r] = 1;
    tb->s[r] = v;
}

static void place_table_sa(oracle_t *o, int32_t t, const int32_t *P, int64_t nP) {
    otab *tb = &o->t[t];
    const int64_t b = o->placements;
    const int32_t W = o->ways;
    const int64_t nslot = tb->nsets * W;
    int64_t nU = tb->have_fwd ? tb->nU : 0, nM = tb->have_fwd ? tb->nM : 0;

    memcpy(tb->way_row0, tb->way_row, sizeof(int32_t) * (size_t)(nslot + 1));
    for (int64_t k = 0; k < nslot; ++k)
        if (tb->way_row0[k] >= 0) tb->in_r0[tb->way_row0[k]] = 1;
#if ORACLE_MUTANT == 15 /* planted: every resident ages once per placement instead of per scan */
    if (o->policy == O_PRIORITY)
        for (int64_t k = 0; k < nslot; ++k)
            if (tb->way_row[k] >= 0) {
                int32_t r = tb->way_row[k];
                tb->s[r] = tb->s[r] > 0 ? tb->s[r] - 1 : 0;
            }
#endif
    /* A. accessed residents: prefetch flag cleared, touch score */
    for (int64_t k = 0; k < nU; ++k) {
        int32_t r = tb->U[k];
        if (tb->in_r[r]) {
            tb->pf[r] = 0;
            tb->s[r] = touch_score(o, tb, r, b);
        }
    }
    /* distinct prefetch rows, ascending */
    int32_t *pd = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nP + 1));
    int64_t npd = 0;
    for (int64_t k = 0; k < nP; ++k)
        if (!tb->in_p[P[k]]) { tb->in_p[P[k]] = 1; pd[npd++] = P[k]; }
    free(tb->lastP);
    tb->lastP = (int32_t *)malloc(sizeof(int32_t) * (size_t)(npd + 1));
    memcpy(tb->lastP, pd, sizeof(int32_t) * (size_t)npd);
    tb->nlastP = npd;
    qsort(pd, (size_t)npd, sizeof(int32_t), cmp_row);
    int32_t *ms = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nM + 1));
    memcpy(ms, tb->M, sizeof(int32_t) * (size_t)nM);
    qsort(ms, (size_t)nM, sizeof(int32_t), cmp_row);
#if ORACLE_MUTANT == 13 /* planted: prefetch events before the misses */
    for (int64_t k = 0; k < npd; ++k) {
        int32_t r = pd[k];
        if (tb->in_r[r]) { if (prefetch_floor(o, tb, r, b) > tb->s[r]) tb->s[r] = prefetch_floor(o, tb, r, b); }
        else sa_insert(o, tb, r, prefetch_score(o, tb, r, b));
    }
    for (int64_t k = 0; k < nM; ++k) if (!tb->in_r[ms[k]]) sa_insert(o, tb, ms[k], touch_score(o, tb, ms[k], b));
#else
    /* B. misses, ascending */
    for (int64_t k = 0; k < nM; ++k) sa_insert(o, tb, ms[k], touch_score(o, tb, ms[k], b));
    /* C. prefetch rows, ascending */
    for (int64_t k = 0; k < npd; ++k) {
        int32_t r = pd[k];
        if (tb->in_r[r]) {
            if (prefetch_floor(o, tb, r, b) > tb->s[r]) tb->s[r] = prefetch_floor(o, tb, r, b);
        } else {
            sa_insert(o, tb, r, prefetch_score(o, tb, r, b));
        }
    }
#endif
    /* counters and prefetch flags */
    int64_t evicted = 0, adm_miss = 0, fill = 0, p_res = 0, p_drop = 0, m_drop = 0;
    for (int64_t k = 0; k < nslot; ++k)
        if (tb->way_row0[k] >= 0 && !tb->in_r[tb->way_row0[k]]) ++evicted;
    uint64_t dig = 0;
    tb->nres = 0;
    for (int64_t k = 0; k < nslot; ++k) {
        int32_t r = tb->way_row[k];
        if (r < 0) continue;
        if (tb->way_row0[k] != r) { /* newly admitted, or moved to another way */
            if (tb->in_m[r]) ++adm_miss; else ++fill;
#if ORACLE_MUTANT == 18
            tb->pf[r] = tb->in_p[r] && !tb->in_m[r];
#else
            tb->pf[r] = tb->in_p[r]; /* R16, as in the fully associative form */
#endif
        }
        tb->res[tb->nres++] = r;
        dig += oracle_splitmix64_mix(((uint64_t)t << 40) | (uint64_t)r);
    }
    for (int64_t k = 0; k < nM; ++k) if (!tb->in_r[ms[k]]) ++m_drop;
    for (int64_t k = 0; k < npd; ++k) {
        if (tb->in_r0[pd[k]]) ++p_res;
        else if (!tb->in_r[pd[k]]) ++p_drop;
    }
    /* clear scratch marks */
    for (int64_t k = 0; k < nslot; ++k)
        if (tb->way_row0[k] >= 0) tb->in_r0[tb->way_row0[k]] = 0;
    for (int64_t k = 0; k < npd; ++k) tb->in_p[pd[k]] = 0;
    for (int64_t k = 0; k < nU; ++k) { tb->in_m[tb->U[k]] = 0; tb->c[tb->U[k]] = 0; }

    tb->plc[0] = evicted; tb->plc[1] = adm_miss; tb->plc[2] = fill; tb->plc[3] = p_res;
    tb->plc[4] = p_drop; tb->plc[5] = m_drop; tb->plc[6] = tb->nres; tb->plc[7] = fill * tb->row_bytes;
    tb->plc[8] = tb->nlastP;
    tb->digest = dig;
    tb->have_fwd = 0;
    tb->have_plc = 1;
    free(pd);
    free(ms);
}

/* ----------------------------------------------------------------- forward */

static void forward_table(oracle_t *o, int32_t t, const int32_t *idx, const int64_t *off, int32_t B,
                          float *out32, double *out64, int64_t out_base) {
    otab *tb = &o->t[t];
    const int64_t *bo = off + (int64_t)t * B;
    int64_t s0 = bo[0], s1 = bo[B], L = s1 - s0;
    /* a forward not followed by a placement leaves marks behind */
    if (tb->have_fwd)
        for (int64_t k = 0; k < tb->nM; ++k) tb->in_m[tb->M[k]] = 0;
    /* distinct rows, hits, misses */
    free(tb->U); free(tb->M); free(tb->last_idx);
    tb->U = (int32_t *)malloc(sizeof(int32_t) * (size_t)(L + 1));
    tb->M = (int32_t *)malloc(sizeof(int32_t) * (size_t)(L + 1));
    tb->last_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(L + 1));
    memcpy(tb->last_idx, idx + s0, sizeof(int32_t) * (size_t)L);
    tb->nlast = L; tb->last_base = s0;
    int64_t nU = 0, nM = 0, hits = 0, hits_pf = 0;
    for (int64_t i = s0; i < s1; ++i) {
        int32_t r = idx[i];
        if (tb->in_u[r]) continue;
        tb->in_u[r] = 1;
        tb->U[nU++] = r;
        if (tb->in_r[r]) { ++hits; if (tb->pf[r]) ++hits_pf; }
        else { tb->M[nM++] = r; tb->in_m[r] = 1; }
    }
    for (int64_t k = 0; k < nU; ++k) tb->in_u[tb->U[k]] = 0;
    tb->nU = nU; tb->nM = nM; tb->have_fwd = 1;
    /* coverage numerator: distinct rows of this batch in set(P) of the
     * placement just before it (none if another forward came between) */
    int64_t covered = 0;
    if (tb->have_plc) {
        for (int64_t k = 0; k < tb->nlastP; ++k) tb->in_p[tb->lastP[k]] = 1;
#if ORACLE_MUTANT == 10 /* planted: lookups counted with their repeats */
        for (int64_t i = s0; i < s1; ++i) covered += tb->in_p[idx[i]];
#else
        for (int64_t k = 0; k < nU; ++k) covered += tb->in_p[tb->U[k]];
#endif
        for (int64_t k = 0; k < tb->nlastP; ++k) tb->in_p[tb->lastP[k]] = 0;
    }
    tb->have_plc = 0;
    tb->fwd[0] = L; tb->fwd[1] = nU; tb->fwd[2] = hits; tb->fwd[3] = hits_pf; tb->fwd[4] = nM;
    tb->fwd[5] = nM * tb->row_bytes; tb->fwd[6] = covered;
    /* pooled sums, double accumulation, one rounding to float */
    for (int32_t j = 0; j < B; ++j) {
        int64_t a = bo[j], e = bo[j + 1];
#if ORACLE_MUTANT == 5 /* planted: the last index of every bag is dropped */
        if (e > a) --e;
#endif
        for (int32_t k = 0; k < tb->d; ++k) {
            double acc = 0.0;
            for (int64_t i = a; i < e; ++i) acc += elem(tb, idx[i], k);
            int64_t p = out_base + (int64_t)j * tb->d + k;
            if (out32) out32[p] = (float)acc;
            if (out64) out64[p] = acc;
        }
    }
}

/* -------------------------------------------------------------- threading */

typedef struct {
    oracle_t *o;
    int32_t first, stride, B;
    int kind; /* 0 placement, 1 forward */
    const int32_t *a;
    const int64_t *off;
    const uint8_t *bits;
    float *out32;
    double *out64;
} job_t;

static void run_table(job_t *j, int32_t t) {
    oracle_t *o = j->o;
    if (j->kind == 0) {
        place_table(o, t, j->a + j->off[t], j->off[t + 1] - j->off[t], j->bits);
    } else {
        int64_t base = 0;
        for (int32_t u = 0; u < t; ++u) base += (int64_t)j->B * o->t[u].d;
        forward_table(o, t, j->a, j->off, j->B, j->out32, j->out64, base);
    }
}

static void *worker(void *arg) {
    job_t *j = (job_t *)arg;
    for (int32_t t = j->first; t < j->o->T; t += j->stride) run_table(j, t);
    return NULL;
}

static void run_all(job_t proto) {
    oracle_t *o = proto.o;
    int32_t nt = o->nthreads < o->T ? o->nthreads : o->T;
    if (nt <= 1) {
        for (int32_t t = 0; t < o->T; ++t) run_table(&proto, t);
        return;
    }
    pthread_t th[256];
    job_t jobs[256];
    if (nt > 256) nt = 256;
    for (int32_t k = 0; k < nt; ++k) {
        jobs[k] = proto; jobs[k].first = k; jobs[k].stride = nt;
        pthread_create(&th[k], NULL, worker, &jobs[k]);
    }
    for (int32_t k = 0; k < nt; ++k) pthread_join(th[k], NULL);
}

/* ---------------------------------------------------------------- entry points */

/* prefetch: table-major rows; poff: [T+1] offsets into it; bits: one byte per
 * access of the most recent forward, or NULL (all zero).  Returns O_E_RANGE
 * (state unchanged) if any prefetch row lies outside its table. */
int32_t oracle_placement(void *h, const int32_t *prefetch, const int64_t *poff, const uint8_t *bits) {
    oracle_t *o = (oracle_t *)h;
    if (!o || !poff) return O_E_INVALID;
    for (int32_t t = 0; t < o->T; ++t) {
        if (poff[t] > poff[t + 1] || poff[0] != 0) return O_E_INVALID;
        for (int64_t k = poff[t]; k < poff[t + 1]; ++k)
            if (prefetch[k] < 0 || prefetch[k] >= o->t[t].n) return O_E_RANGE;
    }
    job_t j = {o, 0, 1, 0, 0, prefetch, poff, bits, NULL, NULL};
    run_all(j);
    o->placements++;
    return O_OK;
}

/* idx: table-major indices; off: [T*B+1] bag offsets; out32 / out64 (either
 * may be NULL): table-major [T][B][D_t]. */
int32_t oracle_forward(void *h, const int32_t *idx, const int64_t *off, int32_t B, float *out32, double *out64) {
    oracle_t *o = (oracle_t *)h;
    if (!o || !off || B < 0) return O_E_INVALID;
    int64_t nb = (int64_t)o->T * B;
    if (off[0] != 0) return O_E_INVALID;
    for (int64_t j = 0; j < nb; ++j) if (off[j + 1] < off[j]) return O_E_INVALID;
    for (int32_t t = 0; t < o->T; ++t)
        for (int64_t i = off[(int64_t)t * B]; i < off[(int64_t)(t + 1) * B]; ++i)
            if (idx[i] < 0 || idx[i] >= o->t[t].n) return O_E_RANGE;
    job_t j = {o, 0, 1, B, 1, idx, off, NULL, out32, out64};
    run_all(j);
    o->forwards++;
    return O_OK;
}

/* L1 mass of every pooled output element: out[t][j][k] = sum over bag j of
 * |E_t[I[i]][k]|, in double (the scale of the pooled-sum tolerance).  Reads
 * only the tables: no cache state, no counters. */
int32_t oracle_pooled_abs(void *h, const int32_t *idx, const int64_t *off, int32_t B, double *out) {
    oracle_t *o = (oracle_t *)h;
    if (!o || !off || !out || B < 0) return O_E_INVALID;
    int64_t base = 0;
    for (int32_t t = 0; t < o->T; ++t) {
        const otab *tb = &o->t[t];
        const int64_t *bo = off + (int64_t)t * B;
        for (int32_t j = 0; j < B; ++j)
            for (int32_t k = 0; k < tb->d; ++k) {
                double acc = 0.0;
                for (int64_t i = bo[j]; i < bo[j + 1]; ++i) {
                    if (idx[i] < 0 || idx[i] >= tb->n) return O_E_RANGE;
                    acc += fabs(elem(tb, idx[i], k));
                }
                out[base + (int64_t)j * tb->d + k] = acc;
            }
        base += (int64_t)B * tb->d;
    }
    return O_OK;
}

/* fwd[7]: lookups, unique, hits, hits_prefetch, misses, ondemand_bytes,
 *         prefetch_covered.
 * plc[9]: evicted, admitted_miss, prefetch_fill, prefetch_resident,
 *         prefetch_dropped, miss_dropped, resident, prefetch_bytes,
 *         prefetch_distinct. */
void oracle_table_stats(void *h, int32_t t, int64_t *fwd, int64_t *plc, uint64_t *digest) {
    oracle_t *o = (oracle_t *)h;
    otab *tb = &o->t[t];
    if (fwd) memcpy(fwd, tb->fwd, sizeof(tb->fwd));
    if (plc) memcpy(plc, tb->plc, sizeof(tb->plc));
    if (digest) *digest = tb->digest;
}

/* Resident rows of table t in ascending order; returns |R| (writes at most
 * `capacity` rows). */
int64_t oracle_resident(void *h, int32_t t, int32_t *rows_out, int64_t capacity) {
    oracle_t *o = (oracle_t *)h;
    otab *tb = &o->t[t];
    int64_t q = 0;
    for (int64_t r = 0; r < tb->n; ++r)
        if (tb->in_r[r]) { if (q < capacity && rows_out) rows_out[q] = (int32_t)r; ++q; }
    return q;
}
