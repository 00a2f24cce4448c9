"""The exact extension solve (tsid_extend_chunk_ridge; Section 5.2, Eq. 6 in
factored form) against the oracle's fp64 normal equations (Cholesky), which
the oracle pins check against numpy's least squares.

The library accumulates each free row's Gram matrix in fp64 on the matrix
cores and factors it in fp64, so the only difference from the oracle is the
order of the fp64 sums and the final rounding of the solution to fp32: each
row must match to a few fp32 ulps (relative error 1e-6 per row), also for
rows with fewer cells than k, whose Gram matrices are singular up to lambda.
"""
import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note

pytestmark = pytest.mark.gpu

ROW_TOL = 1e-6


def _ctx(k):
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    p = synth.random_case(200, 150, 2000, 64, 48, k, seed=5)
    t.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)  # sets the rank
    return t


def _chunk(seed, n_fixed, n_free, nnz, k, hot=0, short=0):
    """Uniform cells plus `hot` fully observed free rows (1 .. hot) and `short`
    free rows with 1 .. k - 1 cells each (after them); free row 0 has none."""
    g = np.random.default_rng(seed)
    F = g.normal(0, k ** -0.25, (n_fixed, k)).astype(np.float32)
    base = g.choice(n_fixed * n_free, min(nnz, n_fixed * n_free), replace=False)
    cells = [base[base % n_free > hot + short]]
    for h in range(hot):
        cells.append(np.arange(n_fixed) * n_free + (1 + h))
    for s in range(short):
        cells.append(g.choice(n_fixed, 1 + s % (k - 1), replace=False) * n_free + (1 + hot + s))
    cells = np.concatenate(cells)
    cells = cells[g.permutation(cells.size)]
    fixed = (cells // n_free).astype(np.int32)
    free = (cells % n_free).astype(np.int32)
    r = g.standard_normal(cells.size).astype(np.float32)
    return F, fixed, free, r


def _run(T, F, fixed, free, r, n_free, lam, side=0):
    import torch
    Fd = torch.from_numpy(F).cuda()
    out = torch.empty((n_free, F.shape[1]), dtype=torch.float32).pin_memory()
    T.extend_chunk(side, fixed, free, r, n_free, Fd, out, float(lam))
    T.sync()
    return out.numpy().copy()


def _row_err(X, Xo):
    X = np.asarray(X, np.float64)
    num = np.linalg.norm(X - Xo, axis=1)
    den = np.maximum(np.linalg.norm(Xo, axis=1), 1e-30)
    return np.where(np.linalg.norm(Xo, axis=1) > 0, num / den, num)


@pytest.mark.parametrize("k", [8, 16, 32, 64, 128])
@pytest.mark.parametrize("lam", [0.5, 1e-3])
def test_ridge_rows_match_oracle(k, lam):
    F, fixed, free, r = _chunk(10 + k, 3000, 600, 50000, k, hot=2, short=40)
    counts = np.bincount(free, minlength=600)
    assert counts[0] == 0 and (counts < k).sum() >= 40 and counts.max() == 3000
    T = _ctx(k)
    try:
        note(f"ridge k={k} lam={lam} nnz={r.size}")
        X = _run(T, F, fixed, free, r, 600, lam)
    finally:
        T.close()
    st, Xo = oracle.ridge(fixed, free, r, 600, F, lam)
    assert st == 0
    err = _row_err(X, Xo)
    assert np.all(X[0] == 0)
    assert err.max() <= ROW_TOL, (err.max(), int(err.argmax()), counts[err.argmax()])


def test_ridge_lambda_zero_full_rank_matches_oracle():
    """lambda = 0 with at least 3k cells per row: the plain least-squares
    solution (the oracle's pin against numpy lstsq)."""
    k = 32
    g = np.random.default_rng(7)
    n_fixed, n_free = 500, 40
    F = g.normal(0, 1.0, (n_fixed, k)).astype(np.float32)
    fixed = np.concatenate([g.choice(n_fixed, 3 * k + f, replace=False) for f in range(n_free)]).astype(np.int32)
    free = np.concatenate([np.full(3 * k + f, f) for f in range(n_free)]).astype(np.int32)
    r = g.standard_normal(fixed.size).astype(np.float32)
    T = _ctx(k)
    try:
        note("ridge lambda=0")
        X = _run(T, F, fixed, free, r, n_free, 0.0)
    finally:
        T.close()
    st, Xo = oracle.ridge(fixed, free, r, n_free, F, 0.0)
    assert st == 0
    assert _row_err(X, Xo).max() <= ROW_TOL


def test_ridge_singular_row_reports_nonfinite():
    """lambda = 0 and a row with fewer cells than k: no unique solution."""
    import paper_2608_00977_amd as tsid
    k = 16
    g = np.random.default_rng(8)
    F = g.normal(0, 1.0, (100, k)).astype(np.float32)
    fixed = g.choice(100, 5, replace=False).astype(np.int32)
    free = np.zeros(5, np.int32)
    r = np.ones(5, np.float32)
    T = _ctx(k)
    try:
        with pytest.raises(tsid.TsidError) as ei:
            _run(T, F, fixed, free, r, 1, 0.0)
        assert ei.value.status == tsid.binding.E_NONFINITE
        # the context stays usable
        X = _run(T, F, fixed, free, r, 1, 0.1)
        st, Xo = oracle.ridge(fixed, free, r, 1, F, 0.1)
        assert st == 0 and _row_err(X, Xo).max() <= ROW_TOL
    finally:
        T.close()


def test_ridge_chunking_is_invariant_and_matches_converged_steps():
    """Rows solved in three chunks in flight equal one chunk bit for bit, and
    the one-sided gradient steps converge to the same solution."""
    import torch
    from paper_2608_00977_amd import make_opts
    k = 32
    F, fixed, free, r = _chunk(21, 400, 90, 9000, k, hot=1, short=10)
    T = _ctx(k)
    try:
        note("ridge chunking")
        whole = _run(T, F, fixed, free, r, 90, 0.5)
        Fd = torch.from_numpy(F).cuda()
        outs = []
        for lo, hi in ((0, 30), (30, 61), (61, 90)):
            m = (free >= lo) & (free < hi)
            out = torch.empty((hi - lo, k), dtype=torch.float32).pin_memory()
            T.extend_chunk(0, fixed[m], (free[m] - lo).astype(np.int32), r[m], hi - lo, Fd, out, 0.5)
            outs.append(out)
        T.sync()
        parts = np.concatenate([o.numpy() for o in outs])
        assert np.array_equal(parts, whole)
        X = torch.empty((90, k), dtype=torch.float32).pin_memory()
        # lr 0.05: a row with one cell has curvature 2 |p|^2 (up to about 20
        # here), so larger steps diverge there
        T.extend_chunk(0, fixed, free, r, 90, Fd, X, make_opts(epochs=6000, lam=0.5, lr=0.05, step="degree"))
        T.sync()
        nz = np.bincount(free, minlength=90) > 0
        rel = np.linalg.norm(X.numpy()[nz] - whole[nz]) / np.linalg.norm(whole[nz])
        assert rel <= 1e-4, rel
    finally:
        T.close()


def test_ridge_rejects_bad_arguments():
    import torch
    import paper_2608_00977_amd as tsid
    T = _ctx(16)
    try:
        F = np.zeros((10, 16), np.float32)
        for lam in (-1.0, float("nan"), float("inf")):
            with pytest.raises(tsid.TsidError) as ei:
                _run(T, F, np.zeros(1, np.int32), np.zeros(1, np.int32), np.ones(1, np.float32), 1, lam)
            assert ei.value.status == tsid.binding.E_INVAL
        # an out-of-range fixed id is found on the device and reported at sync
        Fd = torch.from_numpy(F).cuda()
        out = torch.empty((1, 16), dtype=torch.float32).pin_memory()
        T.extend_chunk(0, np.array([10], np.int32), np.zeros(1, np.int32), np.ones(1, np.float32), 1, Fd,
                       out, 0.1)
        with pytest.raises(tsid.TsidError) as ei:
            T.sync()
        assert ei.value.status == tsid.binding.E_RANGE
    finally:
        T.close()


def test_ridge_extension_end_to_end_matches_oracle():
    """Both extension phases with the exact solve on a Rating-shaped matrix at
    5% scale, against the oracle's ridge solves of the same cells from the
    same template factors (row phase: template columns fixed; column phase:
    every row fixed)."""
    import torch
    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.extension import Extension
    p = synth.rating(scale=0.05)
    lam = 0.05
    g = np.random.default_rng(3)
    Pt = g.normal(0, p.k ** -0.25, (p.I.size, p.k)).astype(np.float32)
    Qt = g.normal(0, p.k ** -0.25, (p.J.size, p.k)).astype(np.float32)
    T = tsid.Tsid(0)
    try:
        T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
        ext = Extension(p.m, p.n, p.u, p.i, p.r, p.I, p.J, n_chunks=4)
        note(f"ridge extension rows={ext.rows.free_ids.size} cols={ext.cols.free_ids.size}")
        P, Q, _ = ext.run(T, torch.from_numpy(Pt).cuda(), torch.from_numpy(Qt).cuda(), lam)
    finally:
        T.close()
    P, Q = P.numpy(), Q.numpy()
    # the oracle: row phase from template-column cells, column phase from all cells
    row_in = np.zeros(p.m, bool)
    row_in[p.I] = True
    col_pos = np.full(p.n, -1, np.int64)
    col_pos[p.J] = np.arange(p.J.size)
    free_rows = ext.rows.free_ids
    rpos = np.full(p.m, -1, np.int64)
    rpos[free_rows] = np.arange(free_rows.size)
    sel = (~row_in[p.u]) & (col_pos[p.i] >= 0)
    st, Pf = oracle.ridge(col_pos[p.i[sel]].astype(np.int32), rpos[p.u[sel]].astype(np.int32), p.r[sel],
                          free_rows.size, Qt, lam)
    assert st == 0
    Pfull = np.zeros((p.m, p.k), np.float64)
    Pfull[p.I] = Pt
    Pfull[free_rows] = Pf
    free_cols = ext.cols.free_ids
    cpos = np.full(p.n, -1, np.int64)
    cpos[free_cols] = np.arange(free_cols.size)
    sel = cpos[p.i] >= 0
    st, Qf = oracle.ridge(p.u[sel].astype(np.int32), cpos[p.i[sel]].astype(np.int32), p.r[sel],
                          free_cols.size, Pfull.astype(np.float32), lam)
    assert st == 0
    # the column phase reads the library's fp32 row factors; the oracle's are
    # its own fp64 ones rounded to fp32, so allow the row error to propagate
    assert _row_err(P[free_rows], Pf).max() <= ROW_TOL
    assert np.linalg.norm(Q[free_cols] - Qf) / np.linalg.norm(Qf) <= 1e-5
    assert np.array_equal(P[p.I], Pt) and np.array_equal(Q[p.J], Qt)
