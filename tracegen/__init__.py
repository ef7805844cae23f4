"""Seeded synthetic workloads for the tiered pooled-embedding lookup.

This module only *draws inputs*: table values, per-batch lookup indices and bag
offsets, prefetch lists and caching bits.  It holds none of the lookup or cache
arithmetic, so both the HIP path and the CPU oracle can be fed from it without
sharing any of the method's code.

The paper measures on Meta's embedding-lookup traces, which are not available
here.  These generators stand in for them, following the access law the paper
states for production traffic: power-law (Zipf) popularity over embedding rows
(Sec. I).  Every random draw is keyed by
``SeedSequence(251108568, spawn_key=(config, table, purpose, batch))`` and
uses the counter-based Philox bit generator, so any batch of any table can be
regenerated independently.

Purposes: 0 values, 1 permutation, 2 pooling, 3 indices, 4 prefetch noise,
5 caching-bit noise, 6 drift, 7 table shape.
"""
from __future__ import annotations

import dataclasses
import math
import os
import threading
from concurrent.futures import ThreadPoolExecutor
from typing import List, Optional, Sequence, Tuple

import numpy as np

ROOT_SEED = 251108568
P_VALUES, P_PERM, P_POOL, P_INDEX, P_PREFETCH, P_BITS, P_DRIFT, P_SHAPE = range(8)

DTYPE_CODES = {"f32": 0, "f16": 1, "bf16": 2}
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2}
NP_STORAGE = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}
POLICY_CODES = {"lru": 0, "priority": 1}

_U64 = np.uint64
_MASK64 = (1 << 64) - 1


_POOL: Optional[ThreadPoolExecutor] = None


def _pmap(fn, items):
    """Map over tables on a thread pool (numpy releases the GIL); results in order.
    Every table draws from streams of its own, so the result does not depend on
    the thread count."""
    global _POOL
    items = list(items)
    if len(items) <= 1:
        return [fn(x) for x in items]
    if _POOL is None:
        _POOL = ThreadPoolExecutor(max_workers=max(1, min(16, os.cpu_count() or 1)))
    return list(_POOL.map(fn, items))


def rng(config: int, table: int, purpose: int, batch: int) -> np.random.Generator:
    """Counter-based generator for one (config, table, purpose, batch) stream."""
    ss = np.random.SeedSequence(ROOT_SEED, spawn_key=(int(config), int(table), int(purpose), int(batch)))
    return np.random.Generator(np.random.Philox(ss))


# ----------------------------------------------------------------------------
# value rounding
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_storage(x64: np.ndarray, dtype: str) -> np.ndarray:
    """Round fp64 draws to the table's storage type (RNE at every step)."""
    if dtype == "f32":
        return x64.astype(np.float32)
    if dtype == "f16":
        return x64.astype(np.float16)
    if dtype == "bf16":
        return f32_to_bf16_bits(x64.astype(np.float32))
    raise ValueError(dtype)


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits_to_f32(a).astype(np.float64)
    return np.asarray(a).astype(np.float64)


# ----------------------------------------------------------------------------
# Feistel row permutation (Black & Rogaway 2002, cycle-walking)
# ----------------------------------------------------------------------------

def _mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output mix (Steele, Lea & Flood 2014), vectorised; used only to
    scramble Feistel round inputs."""
    z = z.astype(_U64, copy=True)
    with np.errstate(over="ignore"):
        z ^= z >> _U64(30)
        z *= _U64(0xBF58476D1CE4E5B9)
        z ^= z >> _U64(27)
        z *= _U64(0x94D049BB133111EB)
        z ^= z >> _U64(31)
    return z


class FeistelPerm:
    """A seeded bijection on [0, n): balanced 4-round Feistel network on the
    smallest even bit width covering n, with cycle-walking back into range."""

    ROUNDS = 4

    def __init__(self, n: int, keys: Sequence[int]):
        self.n = int(n)
        bits = max(2, (self.n - 1).bit_length())
        bits += bits & 1
        self.half = bits // 2
        self.mask = _U64((1 << self.half) - 1)
        self.keys = [_U64(int(k) & _MASK64) for k in keys[: self.ROUNDS]]

    def _enc(self, v: np.ndarray) -> np.ndarray:
        h = _U64(self.half)
        left = v >> h
        right = v & self.mask
        for k in self.keys:
            f = _mix64(right ^ k) & self.mask
            left, right = right, left ^ f
        return (left << h) | right

    def __call__(self, x: np.ndarray) -> np.ndarray:
        y = self._enc(np.asarray(x, dtype=_U64))
        bad = y >= _U64(self.n)
        while bad.any():
            y[bad] = self._enc(y[bad])
            bad = y >= _U64(self.n)
        return y.astype(np.int64)


def make_perm(config: int, table: int, n: int, variant: int = 0) -> FeistelPerm:
    keys = rng(config, table, P_PERM, variant).integers(0, 2**63, size=4, dtype=np.int64)
    return FeistelPerm(n, [int(k) for k in keys])


# ----------------------------------------------------------------------------
# bounded Zipf by inverse CDF
# ----------------------------------------------------------------------------

_CDF_CACHE: dict = {}
_CDF_LOCK = threading.Lock()
_CDF_CACHE_BYTES = 4 << 30


def zipf_cdf(n: int, alpha: float) -> np.ndarray:
    """Cumulative (unnormalised) mass of p_k ∝ k^-alpha for k = 1..n, fp64."""
    key = (int(n), float(alpha))
    with _CDF_LOCK:
        c = _CDF_CACHE.get(key)
        if c is None:
            k = np.arange(1, n + 1, dtype=np.float64)
            c = np.cumsum(k ** (-float(alpha)))
            if sum(v.nbytes for v in _CDF_CACHE.values()) + c.nbytes > _CDF_CACHE_BYTES:
                _CDF_CACHE.clear()
            _CDF_CACHE[key] = c
    return c


def zipf_pmf(n: int, alpha: float) -> np.ndarray:
    k = np.arange(1, n + 1, dtype=np.float64)
    p = k ** (-float(alpha))
    return p / p.sum()


def zipf_ranks(g: np.random.Generator, n: int, alpha: float, size: int) -> np.ndarray:
    """Draw 0-based ranks (k-1) with P(k) ∝ k^-alpha on k in [1, n]."""
    c = zipf_cdf(n, alpha)
    u = g.random(size) * c[-1]
    r = np.searchsorted(c, u, side="right")
    return np.minimum(r, n - 1).astype(np.int64)


# ----------------------------------------------------------------------------
# workload description
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class Table:
    rows: int
    dim: int
    dtype: str       # "f32" | "f16" | "bf16"
    cap: int         # cache slots (rows) in HBM
    alpha: float     # Zipf exponent
    pooling: Tuple   # ("fixed", k) | ("poisson", lam, lo, hi) | ("geometric", mean) | ("onehot",)

    @property
    def row_bytes(self) -> int:
        return self.dim * ELEM_BYTES[self.dtype]


@dataclasses.dataclass
class Workload:
    """One synthetic configuration.  ``prefetch`` is one of
    ("none",), ("exact",), ("replace", frac), ("mix", precise_frac),
    ("headroom", precise_frac)."""
    config: int
    name: str
    tables: List[Table]
    batches: int
    bags: int
    policy: str = "lru"
    eviction_speed: int = 4
    prefetch: Tuple = ("none",)
    drift: Optional[Tuple[int, float]] = None   # (period in batches, fraction of lookups)
    bit_flip: float = 0.17                      # caching-bit noise (PRIORITY configs)
    integer_values: bool = False
    # caching-bit source: ("lookahead",) = reuse in the next two batches with
    # noise; ("optgen", frac, horizon) = Belady-optimal labels (optgen_labels)
    # for a buffer of frac * Cap rows over the first `horizon` batches
    bits: Tuple = ("lookahead",)
    # 0: fully associative caches; W > 0: W-way set-associative caches
    ways: int = 0

    def __post_init__(self):
        self._cache: dict = {}

    @property
    def num_tables(self) -> int:
        return len(self.tables)

    # -- table values ----------------------------------------------------------
    def table_values(self, t: int, out: Optional[np.ndarray] = None, chunk_rows: int = 1 << 16) -> np.ndarray:
        """Values of table t as a [rows, dim] array of its storage type
        (float32, float16, or uint16 bfloat16 bits).  U(-1,1), or integers in
        [-64, 64] when ``integer_values`` is set."""
        tb = self.tables[t]
        if out is None:
            out = np.empty((tb.rows, tb.dim), dtype=NP_STORAGE[tb.dtype])
        assert out.shape == (tb.rows, tb.dim) and out.dtype == NP_STORAGE[tb.dtype]

        def chunk(c0):  # every chunk of rows has a stream of its own
            c1 = min(tb.rows, c0 + chunk_rows)
            g = rng(self.config, t, P_VALUES, c0 // chunk_rows)
            n = (c1 - c0) * tb.dim
            if self.integer_values:
                x = g.integers(-64, 65, size=n).astype(np.float64)
            else:
                x = g.random(n) * 2.0 - 1.0
            out[c0:c1] = to_storage(x, tb.dtype).reshape(c1 - c0, tb.dim)
        _pmap(chunk, range(0, tb.rows, chunk_rows))
        return out

    # -- per-batch trace ---------------------------------------------------------
    def _perm(self, t: int, variant: int = 0) -> FeistelPerm:
        key = ("perm", t, variant)
        p = self._cache.get(key)
        if p is None:
            p = make_perm(self.config, t, self.tables[t].rows, variant)
            self._cache[key] = p
        return p

    def pooling_factors(self, t: int, b: int) -> np.ndarray:
        tb = self.tables[t]
        g = rng(self.config, t, P_POOL, b)
        kind = tb.pooling[0]
        if kind == "fixed":
            return np.full(self.bags, int(tb.pooling[1]), dtype=np.int64)
        if kind == "onehot":
            return np.ones(self.bags, dtype=np.int64)
        if kind == "poisson":
            lam, lo, hi = tb.pooling[1], tb.pooling[2], tb.pooling[3]
            return np.clip(g.poisson(lam, self.bags), lo, hi).astype(np.int64)
        if kind == "geometric":
            return g.geometric(1.0 / float(tb.pooling[1]), self.bags).astype(np.int64)
        raise ValueError(kind)

    def table_indices(self, t: int, b: int, n: int) -> np.ndarray:
        tb = self.tables[t]
        g = rng(self.config, t, P_INDEX, b)
        ranks = zipf_ranks(g, tb.rows, tb.alpha, n)
        rows = self._perm(t)(ranks)
        if self.drift is not None:
            period, frac = self.drift
            e = b // period
            gd = rng(self.config, t, P_DRIFT, b)
            moved = gd.random(n) < frac
            if moved.any():
                rows[moved] = self._perm(t, e + 1)(ranks[moved])
        return rows.astype(np.int32)

    def batch(self, b: int) -> Tuple[np.ndarray, np.ndarray]:
        """(indices int32 [L], offsets int64 [T*B+1]) of batch b, table-major."""
        key = ("batch", b)
        hit = self._cache.get(key)
        if hit is not None:
            return hit
        def one(t):
            pf = self.pooling_factors(t, b)
            return pf, self.table_indices(t, b, int(pf.sum()))
        for t in range(self.num_tables):  # permutations are built once, outside the pool
            self._perm(t)
        parts = _pmap(one, range(self.num_tables))
        lens = np.concatenate([p[0] for p in parts])
        idx_parts = [p[1] for p in parts]
        offsets = np.zeros(lens.size + 1, dtype=np.int64)
        np.cumsum(lens, out=offsets[1:])
        indices = np.concatenate(idx_parts).astype(np.int32) if idx_parts else np.zeros(0, np.int32)
        res = (indices, offsets)
        batch_keys = [k for k in self._cache if k[0] == "batch"]
        if len(batch_keys) > 6:
            del self._cache[min(batch_keys, key=lambda k: k[1])]
        self._cache[key] = res
        return res

    def table_segment(self, offsets: np.ndarray, t: int) -> Tuple[int, int]:
        return int(offsets[t * self.bags]), int(offsets[(t + 1) * self.bags])

    def uniques(self, b: int) -> List[np.ndarray]:
        """Sorted distinct rows per table of batch b (empty for b out of range).
        Used only to draw lookahead prefetch lists and caching bits."""
        if b < 0 or b >= self.batches:
            return [np.zeros(0, np.int32) for _ in self.tables]
        key = ("uniq", b)
        hit = self._cache.get(key)
        if hit is not None:
            return hit
        idx, off = self.batch(b)
        out = _pmap(lambda t: np.unique(idx[slice(*self.table_segment(off, t))]), range(self.num_tables))
        uk = [k for k in self._cache if k[0] == "uniq"]
        if len(uk) > 6:
            del self._cache[min(uk, key=lambda k: k[1])]
        self._cache[key] = out
        return out

    # -- prefetch lists ------------------------------------------------------------
    def prefetch_list(self, b: int) -> Tuple[np.ndarray, np.ndarray]:
        """Prefetch list handed to the placement that precedes forward b:
        (rows int32 [P], offsets int64 [T+1]), table-major; may hold repeats."""
        kind = self.prefetch[0]
        T = self.num_tables
        parts: List[np.ndarray] = []
        if kind == "none":
            parts = [np.zeros(0, np.int32) for _ in range(T)]
        else:
            ub = self.uniques(b)
            ubm1 = self.uniques(b - 1) if kind == "headroom" else None

            def one(t):
                u = ub[t].astype(np.int64)
                n = self.tables[t].rows
                g = rng(self.config, t, P_PREFETCH, b)
                if kind == "exact":
                    p = u
                elif kind == "replace":
                    frac = float(self.prefetch[1])
                    p = u.copy()
                    k = int(math.floor(frac * u.size + 0.5))
                    if k:
                        pos = g.choice(u.size, size=k, replace=False)
                        p[pos] = g.integers(0, n, size=k)
                elif kind == "mix":
                    frac = float(self.prefetch[1])
                    k = int(math.floor(frac * u.size + 0.5))
                    keep = np.sort(g.choice(u.size, size=k, replace=False)) if k else np.zeros(0, np.int64)
                    p = np.concatenate([u[keep], g.integers(0, n, size=u.size - k)])
                elif kind == "headroom":
                    frac = float(self.prefetch[1])
                    h = max(0, self.tables[t].cap - int(ubm1[t].size))
                    length = 2 * h
                    k = min(int(math.floor(frac * length + 0.5)), u.size)
                    keep = np.sort(g.choice(u.size, size=k, replace=False)) if k else np.zeros(0, np.int64)
                    p = np.concatenate([u[keep], g.integers(0, n, size=length - k)])
                else:
                    raise ValueError(kind)
                return p.astype(np.int32)
            parts = _pmap(one, range(T))
        offs = np.zeros(T + 1, dtype=np.int64)
        offs[1:] = np.cumsum([p.size for p in parts])
        rows = np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32)
        return rows, offs

    def warm_list(self, k: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
        """Prefetch list of warm-up placement k of n (placements with no
        forward between them, played before a run that starts in the middle
        of the trace): per table, the rows of Zipf ranks in chunk n-1-k of
        [0, Cap), chunks of ceil(Cap / n) ranks, mapped through the table's
        permutation.  Together the n lists name each table's Cap most popular
        rows once, the most popular chunk last, so the caches start full."""
        T = self.num_tables
        parts = []
        for t in range(T):
            cap = self.tables[t].cap
            step = -(-cap // n) if n > 0 else 0
            j = n - 1 - k
            lo, hi = min(cap, j * step), min(cap, (j + 1) * step)
            parts.append(self._perm(t)(np.arange(lo, hi, dtype=np.int64)).astype(np.int32))
        offs = np.zeros(T + 1, dtype=np.int64)
        offs[1:] = np.cumsum([p.size for p in parts])
        return np.concatenate(parts).astype(np.int32), offs

    # -- caching bits ----------------------------------------------------------------
    def cache_bits(self, b: int) -> Optional[np.ndarray]:
        """One byte per access of batch b: the stand-in for the caching model's
        1-bit output (Sec. V-A).  ("lookahead",): c(r) = [r reused in batch b+1
        or b+2], flipped per distinct row with probability ``bit_flip``.
        ("optgen", frac, horizon): the model's ground truth, OPTgen's label for
        a buffer of frac * Cap rows (Sec. VI-A).  None for LRU configs."""
        if self.policy != "priority":
            return None
        if self.bits[0] == "optgen":
            return self._optgen_bits(b)
        idx, off = self.batch(b)
        fut1, fut2 = self.uniques(b + 1), self.uniques(b + 2)
        out = np.zeros(idx.size, dtype=np.uint8)

        def one(t):
            s, e = self.table_segment(off, t)
            u, inv = np.unique(idx[s:e], return_inverse=True)
            reuse = np.isin(u, fut1[t]) | np.isin(u, fut2[t])
            flip = rng(self.config, t, P_BITS, b).random(u.size) < self.bit_flip
            out[s:e] = (reuse ^ flip).astype(np.uint8)[inv]
        _pmap(one, range(self.num_tables))
        return out


    def _optgen_bits(self, b: int) -> np.ndarray:
        _, frac, horizon = self.bits
        key = ("optgen", frac, horizon)
        labels = self._cache.get(key)
        if labels is None:
            seqs = [[] for _ in self.tables]
            for bb in range(min(horizon, self.batches)):
                for t, u in enumerate(self.uniques(bb)):
                    seqs[t].append(u)
            labels = [optgen_labels(seqs[t], int(math.floor(frac * tb.cap))) for t, tb in enumerate(self.tables)]
            self._cache[key] = labels
        idx, off = self.batch(b)
        out = np.zeros(idx.size, dtype=np.uint8)
        if b >= len(labels[0]):
            return out
        for t in range(self.num_tables):
            s, e = self.table_segment(off, t)
            _, inv = np.unique(idx[s:e], return_inverse=True)
            out[s:e] = labels[t][b][inv]
        return out


def optgen_labels(uniq: List[np.ndarray], capacity: int) -> List[np.ndarray]:
    """Belady-optimal caching labels at batch granularity, after OPTgen (Jain &
    Lin, ISCA 2016), the labeller the paper trains its caching model on
    (Sec. VI-A).

    ``uniq[b]`` holds the sorted distinct rows of batch b of one table.  A row
    used in batch b and next in batch b' asks to stay in the buffer over the
    boundaries b .. b'-1 (boundary k lies between batches k and k+1).  Requests
    are taken in order of b' (the time the reuse happens), and among the same
    b' the shorter ones first, then by row; a request is granted iff every
    boundary it spans still holds fewer than ``capacity`` rows, and then it
    occupies them.  Label 1 marks a granted request: the row should stay until
    its next use (a hit there under the optimal policy); rows with no later
    use in the trace get 0.  Returns one uint8 array per batch, aligned with
    ``uniq[b]``."""
    H = len(uniq)
    labels = [np.zeros(u.size, dtype=np.uint8) for u in uniq]
    if H == 0 or capacity <= 0:
        return labels
    rows = np.concatenate(uniq).astype(np.int64) if H else np.zeros(0, np.int64)
    bats = np.concatenate([np.full(u.size, b, np.int64) for b, u in enumerate(uniq)])
    pos = np.concatenate([np.arange(u.size, dtype=np.int64) for u in uniq])
    order = np.lexsort((bats, rows))  # by row, then batch
    r_s, b_s, p_s = rows[order], bats[order], pos[order]
    same = r_s[1:] == r_s[:-1]  # consecutive uses of one row
    start, end, row, at = b_s[:-1][same], b_s[1:][same], r_s[:-1][same], p_s[:-1][same]
    # requests by (end asc, start desc, row asc)
    o = np.lexsort((row, -start, end))
    start, end, at = start[o], end[o], at[o]
    occ = np.zeros(H, dtype=np.int64)
    i, n = 0, start.size
    while i < n:
        j = i
        while j < n and start[j] == start[i] and end[j] == end[i]:
            j += 1
        a, e = int(start[i]), int(end[i])
        k = min(j - i, max(capacity - int(occ[a:e].max()), 0))
        if k > 0:
            occ[a:e] += k
            lb = labels[a]
            lb[at[i:i + k]] = 1
        i = j
    return labels


# ----------------------------------------------------------------------------
# the five configurations, plus small variants for tests
# ----------------------------------------------------------------------------

def _c3_tables(config: int = 3) -> List[Table]:
    g = rng(config, 0, P_SHAPE, 0)
    tabs = []
    for t in range(26):
        n = int(round(math.exp(g.uniform(math.log(1e3), math.log(2e7)))))
        a = float(g.uniform(0.9, 1.3))
        if t == 0:
            n = 20_000_000
        tabs.append(Table(n, 128, "f16", int(math.floor(0.02 * n)), a, ("poisson", 30.0, 0, 10**9)))
    return tabs


def make_config(cid: int, **overrides) -> Workload:
    """The five configurations at full size (1-based id)."""
    if cid == 1:
        w = Workload(1, "c1", [Table(100_000, 64, "f32", 10_000, 1.05, ("fixed", 20))],
                     batches=100, bags=256, policy="lru", prefetch=("replace", 0.2))
    elif cid == 2:
        w = Workload(2, "c2", [Table(1_000_000, 128, "f32", 50_000, 1.1, ("poisson", 40.0, 1, 200)) for _ in range(8)],
                     batches=500, bags=2048, policy="lru", prefetch=("exact",))
    elif cid == 3:
        w = Workload(3, "c3", _c3_tables(), batches=1000, bags=4096, policy="priority", prefetch=("mix", 0.7))
    elif cid == 4:
        w = Workload(4, "c4", [Table(100_000_000, 128, "bf16", 19_531_250, 1.05, ("fixed", 80)) for _ in range(4)],
                     batches=200, bags=16384, policy="lru", prefetch=("exact",), drift=(50, 0.1))
    elif cid == 5:
        tabs = []
        for t in range(64):
            pool = ("geometric", 25.0) if t < 48 else ("onehot",)
            tabs.append(Table(2_000_000, (32, 64, 128, 256)[t % 4], "f32", 200_000, (0.8, 1.0, 1.2)[t % 3], pool))
        w = Workload(5, "c5", tabs, batches=300, bags=8192, policy="priority", prefetch=("headroom", 0.5))
    else:
        raise ValueError(cid)
    for k, v in overrides.items():
        setattr(w, k, v)
    return w


def scaled_config(cid: int, row_scale: float = 1.0, batches: Optional[int] = None,
                  bags: Optional[int] = None, max_tables: Optional[int] = None, config_id: Optional[int] = None,
                  **overrides) -> Workload:
    """A shape-preserving reduction of configuration ``cid``: rows and cache
    capacity scaled by ``row_scale``; fewer batches, bags or tables.  Seeds are
    keyed by ``config_id`` (default 100 + cid) so reduced runs never alias the
    full-size ones."""
    w = make_config(cid)
    tabs = w.tables[: max_tables] if max_tables else w.tables
    new = []
    for tb in tabs:
        rows = max(8, int(round(tb.rows * row_scale)))
        cap = max(0, min(rows, int(round(tb.cap * row_scale))))
        new.append(dataclasses.replace(tb, rows=rows, cap=cap))
    w2 = Workload(config_id if config_id is not None else 100 + cid, w.name + "_scaled", new,
                  batches=batches or w.batches, bags=bags or w.bags, policy=w.policy,
                  eviction_speed=w.eviction_speed, prefetch=w.prefetch, drift=w.drift, bit_flip=w.bit_flip,
                  ways=w.ways)
    for k, v in overrides.items():
        setattr(w2, k, v)
    return w2


def random_tiny(seed: int, max_rows: int = 16, max_cap: int = 6, max_dim: int = 4, batches: int = 6,
                bags: int = 3, policy: Optional[str] = None, integer_values: bool = True) -> Workload:
    """A tiny random configuration for brute-force and sweep tests."""
    g = np.random.Generator(np.random.Philox(np.random.SeedSequence(ROOT_SEED, spawn_key=(999, seed))))
    T = int(g.integers(1, 4))
    tabs = []
    for _ in range(T):
        n = int(g.integers(1, max_rows + 1))
        cap = int(g.integers(0, max_cap + 1))
        d = int(g.integers(1, max_dim + 1))
        dt = ("f32", "f16", "bf16")[int(g.integers(0, 3))]
        pool = ("poisson", float(g.uniform(0.5, 4.0)), 0, 8)
        tabs.append(Table(n, d, dt, cap, float(g.uniform(0.6, 1.4)), pool))
    pol = policy or ("lru", "priority")[int(g.integers(0, 2))]
    pre = [("none",), ("exact",), ("replace", 0.5), ("mix", 0.5), ("headroom", 0.5)][int(g.integers(0, 5))]
    return Workload(1000 + seed, "tiny", tabs, batches=batches, bags=bags, policy=pol,
                    eviction_speed=int(g.integers(0, 6)), prefetch=pre, integer_values=integer_values)


def expected_unique(n: int, alpha: float, lookups: int) -> float:
    """E[#distinct rows] of ``lookups`` independent Zipf draws: sum_k 1-(1-p_k)^L."""
    p = zipf_pmf(n, alpha)
    return float(np.sum(-np.expm1(lookups * np.log1p(-p))))
