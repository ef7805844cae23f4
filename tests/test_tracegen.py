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
