"""The synthetic workload generator: distributions, bijections, determinism."""
import math

import numpy as np
import pytest
from scipy import stats

import tracegen as tg


@pytest.mark.parametrize("alpha", [0.8, 1.0, 1.3])
def test_zipf_matches_pmf(alpha):
    n, draws = 200, 200_000
    g = tg.rng(7, 0, tg.P_INDEX, 0)
    r = tg.zipf_ranks(g, n, alpha, draws)
    assert r.min() >= 0 and r.max() < n
    obs = np.bincount(r, minlength=n)
    exp = tg.zipf_pmf(n, alpha) * draws
    chi2 = ((obs - exp) ** 2 / exp).sum()
    assert stats.chi2.sf(chi2, n - 1) > 1e-4


@pytest.mark.parametrize("n", [1, 2, 3, 17, 1000, 65537])
def test_feistel_is_bijection(n):
    p = tg.make_perm(3, 1, n)
    y = p(np.arange(n))
    assert np.array_equal(np.sort(y), np.arange(n))


def test_expected_unique_closed_form():
    w = tg.make_config(1)
    seen = [w.uniques(b)[0].size for b in range(20)]
    assert abs(np.mean(seen) - tg.expected_unique(100_000, 1.05, 5120)) < 30


def test_pooling_means():
    w2 = tg.scaled_config(2, row_scale=0.01, bags=4000)
    assert abs(w2.pooling_factors(0, 0).mean() - 40) < 1.0
    w5 = tg.scaled_config(5, row_scale=0.001, bags=4000)
    assert abs(w5.pooling_factors(0, 0).mean() - 25) < 1.5
    assert (w5.pooling_factors(50, 0) == 1).all()
    pf2 = w2.pooling_factors(0, 1)
    assert pf2.min() >= 1 and pf2.max() <= 200


def test_prefetch_fractions():
    w = tg.make_config(1)
    P, poff = w.prefetch_list(3)
    U = w.uniques(3)[0]
    assert P.size == U.size
    k = int(math.floor(0.2 * U.size + 0.5))
    assert U.size - k - 5 <= np.isin(P, U).sum() <= U.size
    w3 = tg.scaled_config(3, row_scale=0.01, batches=4, bags=512, max_tables=3)
    P, poff = w3.prefetch_list(1)
    for t in range(3):
        u = w3.uniques(1)[t]
        assert poff[t + 1] - poff[t] == u.size


def test_determinism_and_ranges():
    a = tg.make_config(2)
    b = tg.make_config(2)
    ia, oa = a.batch(5)
    ib, ob = b.batch(5)
    assert np.array_equal(ia, ib) and np.array_equal(oa, ob)
    assert oa[0] == 0 and oa[-1] == ia.size and (np.diff(oa) >= 0).all()
    for t in range(a.num_tables):
        s, e = a.table_segment(oa, t)
        assert ia[s:e].min() >= 0 and ia[s:e].max() < a.tables[t].rows


def test_bf16_rounding_ties_to_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -2.5], dtype=np.float32)
    b = tg.f32_to_bf16_bits(x)
    back = tg.bf16_bits_to_f32(b)
    assert back.tolist() == [1.0, 1.0, 1.0 + 2**-6, -2.5]


def test_cache_bits_shape():
    w = tg.scaled_config(3, row_scale=0.001, batches=5, bags=256, max_tables=4)
    idx, off = w.batch(1)
    bits = w.cache_bits(1)
    assert bits.shape == idx.shape and set(np.unique(bits)) <= {0, 1}


# ----------------------------------------------------------------------------- OPTgen labels

def _optimal_hits(uniq, capacity):
    """Most hits any demand-filled buffer of `capacity` rows can score on the
    batch sequence (a row hits in batch b if the buffer held it across the
    boundary before b), by exhaustive search over every buffer content."""
    rows = sorted(set().union(*[set(u.tolist()) for u in uniq]))
    idx = {r: i for i, r in enumerate(rows)}
    best = {0: 0}  # buffer content (bit mask) after the previous batch -> hits so far
    for u in uniq:
        used = 0
        for r in u.tolist():
            used |= 1 << idx[r]
        nxt = {}
        for buf, h in best.items():
            h2 = h + bin(buf & used).count("1")
            avail = buf | used  # a row may stay if it was held or was just used
            sub = avail
            while True:  # every subset of avail of at most `capacity` rows
                if bin(sub).count("1") <= capacity and nxt.get(sub, -1) < h2:
                    nxt[sub] = h2
                if sub == 0:
                    break
                sub = (sub - 1) & avail
        best = nxt
    return max(best.values())


@pytest.mark.parametrize("seed", range(40))
def test_optgen_is_optimal_on_tiny_traces(seed):
    g = np.random.default_rng(seed)
    nrows, nb = int(g.integers(2, 7)), int(g.integers(2, 7))
    uniq = [np.unique(g.integers(0, nrows, int(g.integers(0, nrows + 1)))) for _ in range(nb)]
    for cap in range(0, nrows + 1):
        labels = tg.optgen_labels(uniq, cap)
        assert all(l.shape == u.shape for l, u in zip(labels, uniq))
        # a granted request is a hit at the row's next use: the count must be
        # the optimum of an exhaustive search over buffer contents
        assert sum(int(l.sum()) for l in labels) == _optimal_hits(uniq, cap), (seed, cap)
        # the buffer never holds more than cap rows across a boundary
        for k in range(nb - 1):
            held = 0
            for b in range(k + 1):
                for r, lab in zip(uniq[b].tolist(), labels[b].tolist()):
                    nxt = next((bb for bb in range(b + 1, nb) if r in set(uniq[bb].tolist())), None)
                    if lab and nxt is not None and b <= k < nxt:
                        held += 1
            assert held <= cap


def test_optgen_large_and_zero_buffer():
    g = np.random.default_rng(5)
    uniq = [np.unique(g.integers(0, 50, 30)) for _ in range(8)]
    # a buffer that holds every row keeps every row until its next use
    labels = tg.optgen_labels(uniq, 50)
    for b, (u, l) in enumerate(zip(uniq, labels)):
        later = set().union(*[set(x.tolist()) for x in uniq[b + 1:]]) if b + 1 < len(uniq) else set()
        assert l.tolist() == [int(r in later) for r in u.tolist()]
    assert all(int(l.sum()) == 0 for l in tg.optgen_labels(uniq, 0))


def test_optgen_bits_expand_to_accesses():
    w = tg.random_tiny(3, batches=5, policy="priority")
    w.bits = ("optgen", 0.8, 5)
    for b in range(5):
        bits = w.cache_bits(b)
        idx, off = w.batch(b)
        assert bits.shape == idx.shape and bits.dtype == np.uint8
        for t in range(w.num_tables):
            s, e = w.table_segment(off, t)
            for r in np.unique(idx[s:e]):
                assert np.unique(bits[s:e][idx[s:e] == r]).size == 1  # one label per distinct row


def test_configuration_shapes():
    """The five workloads' tables, caches, batches and policies as their recipes state them."""
    w = tg.make_config(1)
    assert [(t.rows, t.dim, t.dtype, t.cap) for t in w.tables] == [(100_000, 64, "f32", 10_000)]
    assert (w.bags, w.batches, w.policy) == (256, 100, "lru")
    w = tg.make_config(2)
    assert w.num_tables == 8 and all((t.rows, t.dim, t.dtype, t.cap) == (1_000_000, 128, "f32", 50_000)
                                     for t in w.tables)
    assert (w.bags, w.batches, w.policy, w.prefetch) == (2048, 500, "lru", ("exact",))
    w = tg.make_config(3)
    assert w.num_tables == 26 and w.tables[0].rows == 20_000_000
    assert all(1_000 <= t.rows <= 20_000_000 and t.dim == 128 and t.dtype == "f16" and t.cap == int(0.02 * t.rows)
               for t in w.tables)
    assert (w.bags, w.batches, w.policy, w.eviction_speed) == (4096, 1000, "priority", 4)
    w = tg.make_config(4)
    # 20 GB of HBM cache over 4 tables of 256-byte rows
    assert w.num_tables == 4 and all((t.rows, t.dim, t.dtype, t.cap) == (100_000_000, 128, "bf16", 19_531_250)
                                     for t in w.tables)
    assert (w.bags, w.batches, w.policy) == (16_384, 200, "lru")
    w = tg.make_config(5)
    assert w.num_tables == 64
    assert [t.dim for t in w.tables[:8]] == [32, 64, 128, 256] * 2
    assert all((t.rows, t.dtype, t.cap) == (2_000_000, "f32", 200_000) for t in w.tables)
    assert (w.bags, w.batches, w.policy) == (8192, 300, "priority")


@pytest.mark.parametrize("n", [1, 3, 7])
def test_warm_lists_name_the_cap_most_popular_rows(n):
    """The n warm-up lists together hold each table's Cap rows of lowest Zipf
    rank (the permutation's images of ranks 0..Cap-1), each exactly once, and
    the last list holds the most popular row."""
    w = tg.scaled_config(5, row_scale=0.005, batches=2, bags=16, max_tables=3)
    lists = [w.warm_list(k, n) for k in range(n)]
    for t, tb in enumerate(w.tables):
        got = np.concatenate([P[o[t]:o[t + 1]] for P, o in lists])
        want = np.sort(w._perm(t)(np.arange(tb.cap)))
        assert got.size == tb.cap and np.array_equal(np.sort(got), want)
        P, o = lists[-1]
        assert int(w._perm(t)(np.zeros(1, np.int64))[0]) in P[o[t]:o[t + 1]]
