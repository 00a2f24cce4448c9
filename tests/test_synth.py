"""Synthetic input generators: determinism, shapes and distributions (CPU)."""
import numpy as np

import tsid_synth as synth


def test_tiny_shape_and_determinism():
    a, b = synth.tiny(), synth.tiny()
    for f in ("u", "i", "r", "tu", "ti", "tr", "I", "J", "P0", "Q0"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    assert a.nnz + a.tu.size == 40000
    assert 0.08 < a.tu.size / 40000 < 0.12
    assert a.I.size == 200 and a.J.size == 160 and np.all(np.diff(a.I) > 0)
    keys = a.u.astype(np.int64) * a.n + a.i
    assert np.unique(keys).size == keys.size
    # unit-variance latent products plus N(0, 0.01) noise
    assert 0.8 < np.var(a.r) < 1.3


def test_holdout_is_a_keyed_hash_of_the_cell():
    u = np.arange(100000, dtype=np.int32) % 977
    i = np.arange(100000, dtype=np.int32) // 977
    m1 = synth.holdout_mask(u, i, 1000, 5)
    perm = np.random.default_rng(0).permutation(u.size)
    m2 = synth.holdout_mask(u[perm], i[perm], 1000, 5)
    assert np.array_equal(m1[perm], m2)
    assert abs(m1.mean() - 0.1) < 0.005
    assert not np.array_equal(m1, synth.holdout_mask(u, i, 1000, 6))


def test_mid_zipf_popularity_and_template():
    p = synth.mid()
    assert p.nnz + p.tu.size == 2_000_000
    keys = p.u.astype(np.int64) * p.n + p.i
    assert np.unique(keys).size == keys.size
    assert set(np.unique(p.r).tolist()) <= {1.0, 2.0, 3.0, 4.0, 5.0}
    deg = np.bincount(p.u, minlength=p.m)
    # most-observed template: degree descending, ids ascending on ties
    d_t = deg[p.I]
    assert np.all(np.diff(d_t) <= 0)
    assert d_t[-1] >= np.sort(deg)[-p.I.size]
    # Zipf column popularity: the rank-frequency slope of the unsaturated
    # middle of the distribution is near -1 on a log-log scale
    cdeg = np.sort(np.bincount(p.i, minlength=p.n))[::-1].astype(float)
    ranks = np.arange(1, cdeg.size + 1)
    sel = slice(200, 3000)
    slope = np.polyfit(np.log(ranks[sel]), np.log(cdeg[sel]), 1)[0]
    assert -1.3 < slope < -0.6


def test_random_case_hot_buckets_in_template():
    p = synth.random_case(40, 30, 200, 10, 8, 4, seed=3, hot_rows=2, hot_cols=1)
    deg = np.bincount(p.u, minlength=p.m)
    assert np.sum(deg[p.I] == p.n) >= 2
    cdeg = np.bincount(p.i, minlength=p.n)
    assert np.sum(cdeg[p.J] == p.m) >= 1
    assert not np.all(np.diff(p.I) > 0)  # local ids follow array order, not sorted


def test_draw_count_solver_matches_the_exact_sum():
    """The binned solver for the number of pairwise draws D: at its D, the exact
    expected count of distinct cells (full double sum) is the target."""
    from tsid_synth.generate import _draws_for_distinct, _zipf_rank_weights
    wr = _zipf_rank_weights(3000, 1.0)
    wc = _zipf_rank_weights(400, 1.0)
    D = _draws_for_distinct(wr, wc, 1.0e5)
    exact = np.sum(-np.expm1(-D * wr[:, None] * wc[None, :]))
    assert abs(exact - 1.0e5) <= 0.01 * 1.0e5


def test_billion_template_cells_follow_the_cell_law():
    """Scaled-down Billion workload: distinct cells inside the template block,
    z-scored values, and each cell observed with probability
    1 - exp(-D w_u w_i) (checked per probability band, both the Bernoulli
    prefix and the Poisson-drawn tail)."""
    from tsid_synth.generate import _zipf_rank_weights
    p = synth.billion_template(scale=0.01)
    q = synth.billion_template(scale=0.01)
    for f in ("u", "i", "r", "tu", "ti", "tr", "I", "J"):
        assert np.array_equal(getattr(p, f), getattr(q, f))
    u = np.concatenate([p.u, p.tu]).astype(np.int64)
    i = np.concatenate([p.i, p.ti]).astype(np.int64)
    r = np.concatenate([p.r, p.tr]).astype(np.float64)
    assert abs(r.mean()) < 1e-3 and abs(r.std() - 1.0) < 1e-3
    rank_u = np.full(p.m, -1)
    rank_u[p.I] = np.arange(p.I.size)
    rank_i = np.full(p.n, -1)
    rank_i[p.J] = np.arange(p.J.size)
    a, b = rank_u[u], rank_i[i]
    assert np.all(a >= 0) and np.all(b >= 0)
    keys = a * p.J.size + b
    assert np.unique(keys).size == keys.size
    assert 0.07 < p.tu.size / keys.size < 0.13
    wr = _zipf_rank_weights(p.m, 1.0)[: p.I.size]
    wc = _zipf_rank_weights(p.n, 1.0)[: p.J.size]
    prob = -np.expm1(-p.extra["draws"] * wr[:, None] * wc[None, :])
    seen = np.zeros(prob.shape, dtype=bool)
    seen[a, b] = True
    assert abs(seen.sum() - prob.sum()) <= 5 * np.sqrt(prob.sum())
    for lo, hi in ((0.01, 0.05), (0.05, 0.2), (0.2, 0.5), (0.5, 0.8), (0.8, 0.99)):
        band = (prob >= lo) & (prob < hi)
        mean_p = prob[band].mean()
        sd = np.sqrt(np.sum(prob[band] * (1 - prob[band]))) / band.sum()
        assert abs(seen[band].mean() - mean_p) <= 5 * sd + 1e-3, (lo, hi)


def test_similarity_graph_is_symmetric_and_simple():
    r, c, v = synth.similarity_graph(500, 8, 3)
    assert r.size == c.size == v.size > 0
    assert np.all(r != c) and np.all((v > 0) & (v <= 1))
    key = r.astype(np.int64) * 500 + c
    assert np.unique(key).size == key.size
    fw = dict(zip(key.tolist(), v.tolist()))
    assert all(fw[int(b) * 500 + int(a)] == w for a, b, w in zip(r, c, v))
    r2, c2, v2 = synth.similarity_graph(500, 8, 3)
    assert np.array_equal(r, r2) and np.array_equal(v, v2)
