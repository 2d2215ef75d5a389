"""The seeded generator makes what its recipe says (sizes, moments, skew) and is a
pure function of (seed, counter)."""
import math

import numpy as np
import pytest


def test_tiny_workload(gen):
    w = gen.workload("tiny")
    tr, te = gen.make(w)
    assert len(tr) == 49_500 and len(te) == 500
    cells = np.concatenate([tr["u"].astype(np.int64) * w["n"] + tr["v"], te["u"].astype(np.int64) * w["n"] + te["v"]])
    assert len(np.unique(cells)) == 50_000  # distinct cells
    assert tr["u"].min() >= 0 and tr["u"].max() < w["m"] and tr["v"].max() < w["n"]
    r = tr["r"].astype(np.float64)
    # r = p*.q* + N(0, 0.1): mean 0, variance 1 + 0.1
    assert abs(r.mean()) < 0.03 and r.var() == pytest.approx(1.1, rel=0.03)
    tr2, te2 = gen.make(w)
    assert np.array_equal(tr, tr2) and np.array_equal(te, te2)


def test_planted_factor_moments(gen):
    w = gen.workload("netflix", m=20000, n=3000)
    Ps, Qs = gen.planted(w)
    var = 1 / math.sqrt(128)
    assert float(Ps.var()) == pytest.approx(var, rel=0.01) and abs(float(Ps.mean())) < 2e-3
    assert float(Qs.var()) == pytest.approx(var, rel=0.01)


def test_netflix_shaped_ratings_and_skew(gen):
    w = gen.workload("netflix", ntrain=1_000_000, ntest=1000)
    tr, te = gen.make(w)
    r = tr["r"]
    assert set(np.unique(r).tolist()) <= {1.0, 2.0, 3.0, 4.0, 5.0}
    assert 3.3 < float(r.mean()) < 3.8
    # Zipf(1.0): the most popular rank has probability 1/H_N
    for col, N in (("u", w["m"]), ("v", w["n"])):
        H = float(np.sum(1.0 / np.arange(1, N + 1)))
        top = np.bincount(tr[col], minlength=N).max() / len(tr)
        assert top == pytest.approx(1.0 / H, rel=0.03)


def test_zipf_slope(gen):
    cdf, perm = gen.zipf_table(5000, 0.8, 123, 0)
    pmf = np.diff(np.concatenate([[0.0], cdf]))
    ranks = np.arange(1, 5001)
    slope = np.polyfit(np.log(ranks), np.log(pmf), 1)[0]
    assert slope == pytest.approx(-0.8, abs=1e-6)
    assert sorted(perm.tolist()) == list(range(5000))


def test_counter_draws_are_chunk_invariant(gen):
    w = gen.workload("yahoo", m=5000, n=4000, ntrain=10000, ntest=0)
    a = gen.draw(w, 0, 10000)
    b = np.concatenate([gen.draw(w, 0, 3000), gen.draw(w, 3000, 7000)])
    assert np.array_equal(a, b)
    assert a["r"].min() >= 0 and a["r"].max() <= 5.0
    assert np.allclose(a["r"] * 20, np.round(a["r"] * 20))


def test_hugewiki_shape_items_uniform(gen):
    w = gen.workload("hugewiki", m=200_000, ntrain=400_000, ntest=0)
    a = gen.draw(w, 0, 400_000)
    cv = np.bincount(a["v"], minlength=w["n"])
    # uniform items: counts ~ Poisson(10)
    assert cv.mean() == pytest.approx(400_000 / w["n"]) and cv.max() < 40
    assert abs(float(a["r"].mean())) < 0.02 and float(a["r"].var()) == pytest.approx(2.0, rel=0.03)


def test_guided_zipf_pick_equals_plain_search(gen):
    N, a, seed = 3_000_000, 1.0, 77
    bits = gen.guide_bits(N)
    rng = np.random.default_rng(5)
    G = 1 << bits
    j = rng.integers(0, G, 20_000)
    edges = np.concatenate([j / G, np.nextafter(j / G, 0.0), np.nextafter(j / G, 1.0), [0.0, np.nextafter(1.0, 0.0)]])
    cdf, _ = gen.zipf_table(N, a, seed, 0)
    x = np.concatenate([rng.random(200_000), edges, cdf[:1000], np.nextafter(cdf[:1000], 0.0)])
    x = x[(x >= 0) & (x < 1)]
    assert np.array_equal(gen.pick(x, N, a, seed, 0, guided=True), gen.pick(x, N, a, seed, 0, guided=False))
    w = gen.workload("yahoo", ntrain=200_000, ntest=0)
    assert np.array_equal(gen.draw(w, 0, 200_000), gen.draw(w, 0, 200_000, guided=False))


def test_hugewiki_planted_rank(gen):
    w = gen.workload("hugewiki", m=100_000, ntrain=300_000, ntest=0)
    Ps, Qs = gen.planted(w)
    assert Ps.shape == (100_000, 16) and Qs.shape == (w["n"], 16)
    assert float(Ps.var()) == pytest.approx(1 / math.sqrt(16), rel=0.01)


def test_yahoo_shaped_ratings(gen):
    """r = clamp(round(100 Phi(p*.q* + N(0, 0.25))), 0, 100) / 20: integer
    percentiles over 0..100 (divided by 20), symmetric about 50 since
    p*.q* + noise has mean 0, and heavier at the ends than a uniform because
    its variance (1.25) exceeds the standard normal's."""
    w = gen.workload("yahoo", m=20_000, n=15_000, ntrain=400_000, ntest=0)
    r = gen.draw(w, 0, w["ntrain"])["r"].astype(np.float64) * 20  # r is stored in binary32
    assert np.allclose(r, np.round(r), atol=1e-4) and r.min() >= 0 and r.max() <= 100
    r = np.round(r)
    h = np.bincount(r.astype(np.int64), minlength=101)
    assert h[0] > 0 and h[100] > 0
    assert abs(r.mean() - 50) < 1.0
    # P(percentile <= 10) = P(Z * sqrt(1.25) <= Phi^-1(0.105)) ~ 0.13 > 0.105 (uniform)
    assert 0.12 < h[:11].sum() / len(r) < 0.145
