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


def test_scientific_stream_partitions_the_matrix():
    """Template block + row phase + column phase of the streamed Scientific
    matrix are exactly the training cells of a brute-force pass over every
    cell with the generator's two hash tests, and the C generator reproduces
    the template block's cells and values."""
    from tsid_synth.generate import _cell_hash, _hash_below, holdout_mask
    from tsid_synth.stream import _p, lib
    p = synth.scientific_template(side=192, m=2500)
    om = synth.omega_outside_template(p)
    rows, cols = om.row_phase(), om.col_phase()
    uu, ii = np.meshgrid(np.arange(p.m, dtype=np.uint64), np.arange(p.n, dtype=np.uint64), indexing="ij")
    train = _hash_below(_cell_hash(uu, ii, p.n, 4, "cells"), 0.1) & ~holdout_mask(uu, ii, p.n, 4)
    assert rows.nnz + cols.nnz + p.nnz == int(train.sum())
    # the row phase's cells of each free row are its training cells in the template columns
    a, fl, _ = rows.cells(np.arange(0, rows.free_ids.size, 97))
    for f in np.unique(fl)[:5]:
        u = rows.free_ids[f]
        want = np.flatnonzero(train[u, p.J])  # template positions
        assert np.array_equal(np.sort(a[fl == f]), want)
    # the column phase's cells of a free column: every training row
    a, fl, _ = cols.cells([3])
    assert np.array_equal(a, np.flatnonzero(train[:, cols.free_ids[3]]))
    # the template block through the C generator equals the Python generator's
    I, J = np.ascontiguousarray(p.I, np.int32), np.ascontiguousarray(p.J, np.int32)
    cnt = np.empty(I.size, np.int64)
    lib().sci_count(1, _p(I), I.size, _p(J), J.size, p.n, *om.keys, _p(cnt))
    off = np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)
    f, fl, r = (np.empty(off[-1], t) for t in (np.int32, np.int32, np.float32))
    lib().sci_fill(1, _p(I), I.size, _p(J), J.size, 1, p.n, *om.keys, _p(om.A), _p(om.Bs), p.k, _p(off), _p(f),
                   _p(fl), _p(r))
    kc = I[fl].astype(np.int64) * p.n + f
    kp = p.u.astype(np.int64) * p.n + p.i
    oc, op = np.argsort(kc), np.argsort(kp)
    assert np.array_equal(kc[oc], kp[op])
    np.testing.assert_allclose(r[oc], p.r[op], rtol=1e-5, atol=1e-5)


def test_billion_stream_is_consistent_and_reproducible():
    """The streamed Billion-scale cells: fixed ids in range, free lines
    outside the template, values z-scored with the template's scale, any
    range of lines generated alone gives the same cells, and the template
    block plus both phases hold about the matrix's expected cells."""
    p = synth.billion_template(scale=0.02)
    om = synth.omega_outside_template(p)
    rows, cols = om.row_phase(), om.col_phase()
    assert not np.isin(rows.free_ids, p.I).any() and not np.isin(cols.free_ids, p.J).any()
    total = (rows.nnz + cols.nnz + p.nnz) / 0.9
    assert abs(total / (1e9 * 0.02 * 0.02) - 1.0) < 0.05
    for ph, n_fixed in ((rows, p.J.size), (cols, p.m)):
        fx, fl, r = (np.empty(ph.nnz, t) for t in (np.int32, np.int32, np.float32))
        assert ph.fill(0, ph.free_ids.size, fx, fl, r) == ph.nnz
        assert fx.min() >= 0 and fx.max() < n_fixed
        assert np.array_equal(np.bincount(fl, minlength=ph.free_ids.size), ph.counts)
        assert np.all(np.diff(fl) >= 0)
        assert abs(r.mean()) < 0.1 and abs(r.std() - 1.0) < 0.1
        lines = np.array([1, 7, ph.free_ids.size - 1])
        a, f2, v = ph.cells(lines)
        for ln in lines:
            assert np.array_equal(a[f2 == ln], fx[fl == ln]) and np.array_equal(v[f2 == ln], r[fl == ln])
        # no repeated cell within a line
        key = fl.astype(np.int64) * (n_fixed + 1) + fx
        assert np.unique(key).size == key.size
