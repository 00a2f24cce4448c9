"""Pins of the fp64 CPU oracle to facts fixed by the paper and by mathematics,
independent of the oracle's own code (CPU only).

Each test names what it pins and why a plausible mistake in the oracle (a
dropped term, a wrong sign or index, a transposed operand, a Gauss-Seidel
instead of a Jacobi sweep) would fail it.
"""
import json
import math
import os

import numpy as np
import pytest

import tsid_synth as synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _full_cells(m, n):
    a, b = np.nonzero(np.ones((m, n)))
    return a.astype(np.int32), b.astype(np.int32)


# ---------------------------------------------------------------- P0 golden
def test_hand_derived_steps(oracle_lib):
    """Single epochs derived by hand from Eqs. 2-5 and the clip of Section 5.3."""
    g = json.load(open(os.path.join(GOLDEN, "hand_steps.json")))
    one = np.zeros(1, np.int32)
    for c in g["cases"]:
        st, P, Q, h, _ = oracle_lib.fit(one, one, np.array([c["r"]], np.float32),
                                        np.array([[c["p"]]]), np.array([[c["q"]]]), 1,
                                        c["lambda"], c["lr"], c["step"], c["clip"], c["xi"])
        assert st == 0, c["name"]
        assert h[0] == pytest.approx(c["loss0"], rel=1e-15), c["name"]
        assert P[0, 0] == pytest.approx(c["p1"], rel=1e-14), c["name"]
        assert Q[0, 0] == pytest.approx(c["q1"], rel=1e-14), c["name"]
    t = g["two_cells"]
    cells = np.array(t["cells"])
    st, P, Q, h, _ = oracle_lib.fit(cells[:, 0].astype(np.int32), cells[:, 1].astype(np.int32),
                                    cells[:, 2].astype(np.float32), np.array(t["P"]),
                                    np.array(t["Q"]), 1, t["lambda"], t["lr"], "degree")
    assert st == 0
    assert h[0] == pytest.approx(t["loss0"], rel=1e-15)
    np.testing.assert_allclose(P, t["P1"], rtol=1e-14)
    np.testing.assert_allclose(Q, t["Q1"], rtol=1e-14)


def test_hand_derived_step_scale_and_clip_order(oracle_lib):
    """Rows and columns of degree 2 where the clip acts between D/n and D:
    the clip after the step scale (clip 1), the clip before it (clip 3, the
    order Section 5.3 prints), the degree step on both sides and on the
    columns only (Eq. 5 as printed) all end at different factors, each
    derived by hand.  Swapping the clip and the 1/n, or scaling the wrong
    side, fails one of these cases."""
    g = json.load(open(os.path.join(GOLDEN, "hand_steps.json")))["two_lines"]
    cells = np.array(g["cells"])
    a, b, v = cells[:, 0].astype(np.int32), cells[:, 1].astype(np.int32), cells[:, 2].astype(np.float32)
    seen = set()
    for c in g["cases"]:
        st, P, Q, h, _ = oracle_lib.fit(a, b, v, np.array(g["P"]), np.array(g["Q"]), 1, c["lambda"], g["lr"],
                                        c["step"], c["clip"], c["xi"])
        assert st == 0, c["name"]
        assert h[0] == pytest.approx(c["loss0"], rel=1e-15), c["name"]
        np.testing.assert_allclose(P, c["P1"], rtol=1e-15, err_msg=c["name"])
        np.testing.assert_allclose(Q, c["Q1"], rtol=1e-15, err_msg=c["name"])
        seen.add((c["lambda"], tuple(np.ravel(c["P1"])), tuple(np.ravel(c["Q1"]))))
    assert len(seen) == len(g["cases"])  # every option pair ends elsewhere


def test_hand_derived_bf16_epoch(oracle_lib):
    """bf16 mode (reading R13): the products read round-to-nearest-even bf16
    copies while the fp64 master takes the update and enters the regulariser
    and the loss norms.  The start values straddle bf16 rounding boundaries,
    so rounding the master, using the copy in the regulariser or the master
    in the products each moves p1 or q1 by more than 1e-4."""
    c = json.load(open(os.path.join(GOLDEN, "hand_steps.json")))["bf16"]
    one = np.zeros(1, np.int32)
    st, P, Q, h, _ = oracle_lib.fit(one, one, np.array([c["r"]], np.float32), np.array([[c["p"]]]),
                                    np.array([[c["q"]]]), 1, c["lambda"], c["lr"], c["step"], c["clip"], c["xi"],
                                    bf16=True)
    assert st == 0
    assert h[0] == pytest.approx(c["loss0"], rel=1e-15)
    assert P[0, 0] == pytest.approx(c["p1"], rel=1e-15)
    assert Q[0, 0] == pytest.approx(c["q1"], rel=1e-15)
    # the fp64 run from the same start differs (the bf16 copies matter)
    _, P64, _, _, _ = oracle_lib.fit(one, one, np.array([c["r"]], np.float32), np.array([[c["p"]]]),
                                     np.array([[c["q"]]]), 1, c["lambda"], c["lr"], c["step"], c["clip"], c["xi"])
    assert abs(P64[0, 0] - c["p1"]) > 1e-4


def test_column_only_step_and_printed_clip_are_not_extension_options(oracle_lib):
    """The extension scales the free rows by their own degree (reading R12):
    the column-only step is a template-fit option and returns 1; clip 3 runs."""
    fixed = np.array([0, 1, 0], np.int32)
    free = np.array([0, 0, 1], np.int32)
    v = np.array([1.0, 2.0, 3.0], np.float32)
    F = np.array([[1.0, 0.0], [0.0, 1.0]])
    assert oracle_lib.extend(fixed, free, v, 2, F, 3, 0.0, 0.1, "col_degree")[0] == 1
    st, X3 = oracle_lib.extend(fixed, free, v, 2, F, 1, 0.0, 0.5, "degree", "printed", 0.5)
    # free row 0: D = 2 (1*[1,0] + 2*[0,1]) = [2, 4], deg 2 -> d = (1/2) min(D, 0.5) = [0.25, 0.25]
    # free row 1: D = 2*3*[1,0] = [6, 0], deg 1 -> d = [0.5, 0]
    assert st == 0
    np.testing.assert_allclose(X3, [[0.125, 0.125], [0.25, 0.0]], rtol=1e-15)


@pytest.mark.parametrize("case", ["tiny_sum", "ragged_degree_clip", "ragged_col_printed_bf16", "nonfinite"])
def test_line_parallel_fit_is_the_serial_fit_bit_for_bit(oracle_lib, case):
    """or_fit_lines (rows, then columns, split across OpenMP threads; the
    all-core CPU baseline and the oracle of the largest workloads) gives the
    same bits as the serial or_fit: every sum has the same operands in the
    same order."""
    if case == "tiny_sum":
        p = synth.tiny()
        opts = dict(step="sum", clip=False, bf16=False, lr=p.lr, epochs=6)
    else:
        p = synth.random_case(700, 500, 9000, 300, 200, 32, seed=71, hot_rows=3, hot_cols=2)
        opts = {"ragged_degree_clip": dict(step="degree", clip=True, bf16=False, lr=0.1, epochs=5),
                "ragged_col_printed_bf16": dict(step="col_degree", clip="printed", bf16=True, lr=0.01, epochs=5),
                "nonfinite": dict(step="sum", clip=False, bf16=False, lr=1e5, epochs=40)}[case]
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    ref = oracle_lib.fit(a, b, v, p.P0, p.Q0, opts["epochs"], p.lam, opts["lr"], opts["step"], opts["clip"], 0.05,
                         bf16=opts["bf16"])
    for omp in (True, False):
        got = oracle_lib.fit_lines(a, b, v, p.P0, p.Q0, opts["epochs"], p.lam, opts["lr"], opts["step"], opts["clip"],
                                   0.05, bf16=opts["bf16"], omp=omp)
        assert got[0] == ref[0] and got[4] == ref[4]
        assert np.array_equal(got[1], ref[1]) and np.array_equal(got[2], ref[2])
        assert np.array_equal(got[3], ref[3], equal_nan=True)
    if case == "nonfinite":
        assert ref[0] == 7
    assert oracle_lib.threads(True) >= 1 and oracle_lib.threads(False) == 1


# ------------------------------------------------------------ P1 gradient
@pytest.mark.parametrize("step", ["sum", "degree"])
def test_gradient_matches_central_differences(oracle_lib, step):
    """Eqs. 3-4 summed over Omega* plus 2*lambda*x is the gradient of Eq. 2.
    L is quadratic in any single coordinate, so a central difference of the
    loss is exact up to rounding.  The gradient is read back from one oracle
    epoch, (x0 - x1) / lr (times the degree for the degree step); the Q part
    must be taken at (P_t, Q_t), which pins the simultaneous (Jacobi) update."""
    p = synth.random_case(9, 7, 30, 9, 7, 3, seed=21, lam=0.3)
    a, b, v = p.u, p.i, p.r  # template = everything (I, J are permutations)
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    P0 = p.P0.astype(np.float64)
    Q0 = p.Q0.astype(np.float64)
    lr = 1e-3
    st, P1, Q1, h, _ = oracle_lib.fit(a, b, v, P0, Q0, 1, p.lam, lr, step)
    assert st == 0
    deg_r = np.bincount(a, minlength=P0.shape[0]).clip(1, None)[:, None]
    deg_c = np.bincount(b, minlength=Q0.shape[0]).clip(1, None)[:, None]
    gP = (P0 - P1) / lr
    gQ = (Q0 - Q1) / lr
    if step == "degree":
        gP *= deg_r
        gQ *= deg_c
    h_ = 1e-3
    for X, G, isP in ((P0, gP, True), (Q0, gQ, False)):
        for idx in np.ndindex(*X.shape):
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += h_
            Xm[idx] -= h_
            if isP:
                Lp = oracle_lib.loss(a, b, v, P0.shape[0], Q0.shape[0], Xp, Q0, p.lam)
                Lm = oracle_lib.loss(a, b, v, P0.shape[0], Q0.shape[0], Xm, Q0, p.lam)
            else:
                Lp = oracle_lib.loss(a, b, v, P0.shape[0], Q0.shape[0], P0, Xp, p.lam)
                Lm = oracle_lib.loss(a, b, v, P0.shape[0], Q0.shape[0], P0, Xm, p.lam)
            fd = (Lp - Lm) / (2 * h_)
            assert abs(fd - G[idx]) <= 1e-8 * max(1.0, abs(fd)), (isP, idx, fd, G[idx])
    # the recorded loss is Eq. 2 at (P0, Q0), with the regularisation once per row
    direct = sum((float(v[e]) - P0[a[e]] @ Q0[b[e]]) ** 2 for e in range(v.size))
    direct += p.lam * ((P0 ** 2).sum() + (Q0 ** 2).sum())
    assert h[0] == pytest.approx(direct, rel=1e-13)


# ------------------------------------------------------- P2 closed form optimum
def test_fully_observed_optimum_is_singular_value_soft_threshold(oracle_lib):
    """Fully observed R (6 x 5), rank-k factors:  min ||R - P Q^T||^2 +
    lambda(||P||^2 + ||Q||^2) equals min over rank<=k X of ||R - X||^2 +
    2 lambda ||X||_*, solved by soft-thresholding the top k singular values at
    lambda.  Optimal value and minimiser checked against numpy's SVD."""
    g = np.random.default_rng(5)
    R = g.standard_normal((6, 5)).astype(np.float32).astype(np.float64)
    a, b = _full_cells(6, 5)
    v = R[a, b].astype(np.float32)
    U, S, Vt = np.linalg.svd(R)
    k, lam = 3, 0.1
    Lstar = sum(2 * lam * s - lam * lam if s > lam else s * s for s in S[:k]) + (S[k:] ** 2).sum()
    X = U[:, :k] @ np.diag(np.maximum(S[:k] - lam, 0)) @ Vt[:k]
    P0 = g.normal(0, 0.5, (6, k))
    Q0 = g.normal(0, 0.5, (5, k))
    st, P, Q, h, _ = oracle_lib.fit(a, b, v, P0, Q0, 3000, lam, 0.02, "sum")
    assert st == 0
    assert abs(h[-1] - Lstar) <= 1e-10 * Lstar
    np.testing.assert_allclose(P @ Q.T, X, atol=1e-8)


# ------------------------------------------------------ P3 least squares
def test_extension_matches_least_squares(oracle_lib):
    """With the fixed side held constant (Section 5.2, Eq. 6 in factored
    form) each free row is a ridge regression: x = argmin sum (r - p.x)^2 +
    lambda ||x||^2, i.e. the least-squares solution of [P_obs; sqrt(lambda) I]
    x = [r; 0].  Both the gradient iteration and the Cholesky solve must reach
    numpy.linalg.lstsq of that stacked system."""
    g = np.random.default_rng(9)
    m, n, k, lam = 6, 5, 3, 0.05
    F = g.standard_normal((m, k))
    R = g.standard_normal((m, n)).astype(np.float32)
    mask = g.random((m, n)) < 0.8
    mask[:, 0] = True
    fixed, free = np.nonzero(mask)
    v = R[fixed, free]
    st, Xgd = oracle_lib.extend(fixed, free, v, n, F, 4000, lam, 0.3, "degree")
    assert st == 0
    st, Xch = oracle_lib.ridge(fixed, free, v, n, F, lam)
    assert st == 0
    for f in range(n):
        rows = fixed[free == f]
        A = np.vstack([F[rows], math.sqrt(lam) * np.eye(k)])
        y = np.concatenate([R[rows, f].astype(np.float64), np.zeros(k)])
        x = np.linalg.lstsq(A, y, rcond=None)[0]
        np.testing.assert_allclose(Xch[f], x, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(Xgd[f], x, rtol=1e-8, atol=1e-10)


def _adam_case(seed, n_b=6, k=3, n_free=3, n_fixed=9):
    g = np.random.default_rng(seed)
    F = g.standard_normal((n_fixed, k))
    B = g.standard_normal((n_b, k))
    fixed, free = np.nonzero(g.random((n_fixed, n_free)) < 0.8)
    v = g.standard_normal(fixed.size).astype(np.float32)
    return F, B, fixed.astype(np.int32), free.astype(np.int32), v


def test_extension_adam_first_step_is_normalised_gradient(oracle_lib):
    """Stage II as Eq. 6 states it, Adam on the coefficients C (Section 5.2).
    From C = 0 the gradient of L(C) is G_f = -2 sum r B p (the predictions are
    zero), and after the bias correction Adam's first step is exactly
    -lr G / (|G| + eps) elementwise, whatever beta1 and beta2 are.  A dropped
    bias correction, a transposed basis or a wrong sign fails this."""
    F, B, fixed, free, v = _adam_case(31)
    lr, eps = 0.01, 1e-8
    for b1, b2 in ((0.9, 0.999), (0.5, 0.9)):
        st, X, C1 = oracle_lib.extend_adam(fixed, free, v, 3, F, B, 1, 0.2, lr, b1, b2, eps)
        assert st == 0
        for f in range(3):
            sel = free == f
            G = -2.0 * B @ (F[fixed[sel]].T @ v[sel].astype(np.float64))
            np.testing.assert_allclose(C1[f], -lr * G / (np.abs(G) + eps), rtol=1e-12, atol=1e-15)
            np.testing.assert_allclose(X[f], B.T @ C1[f], rtol=1e-12, atol=1e-15)


def test_extension_adam_without_moments_is_sign_descent(oracle_lib):
    """With beta1 = beta2 = 0 and eps = 0 the moment estimates are the current
    gradient and its square, so each Adam step is C <- C - lr sign(dL/dC): the
    textbook sign-gradient method, run here from the loss's own gradient
    (least squares in the coefficients, with the design rows B p)."""
    F, B, fixed, free, v = _adam_case(32)
    lam, lr, steps = 0.3, 0.02, 7
    st, _, C = oracle_lib.extend_adam(fixed, free, v, 3, F, B, steps, lam, lr, 0.0, 0.0, 0.0)
    assert st == 0
    for f in range(3):
        sel = free == f
        A = F[fixed[sel]] @ B.T          # design rows: prediction = A c
        y = v[sel].astype(np.float64)
        c = np.zeros(B.shape[0])
        for _ in range(steps):
            grad = -2.0 * A.T @ (y - A @ c) + 2.0 * lam * c
            c = c - lr * np.sign(grad)
        np.testing.assert_allclose(C[f], c, rtol=1e-12, atol=1e-14)


def test_extension_adam_converges_to_coefficient_ridge(oracle_lib):
    """Many small Adam steps reach the minimiser of L(C), a ridge regression in
    the coefficients: c_f = argmin ||A c - r||^2 + lambda ||c||^2 with design
    rows A = (B p)^T, solved here by numpy.linalg.lstsq of the stacked system
    [A; sqrt(lambda) I] c = [r; 0].  (Its factor B^T c_f differs from the
    factored extension's: the penalty is on C, not on B^T C.)"""
    F, B, fixed, free, v = _adam_case(33)
    lam = 0.3
    st, X, C = oracle_lib.extend_adam(fixed, free, v, 3, F, B, 30000, lam, 2e-3)
    assert st == 0
    for f in range(3):
        sel = free == f
        A = F[fixed[sel]] @ B.T
        M = np.vstack([A, math.sqrt(lam) * np.eye(B.shape[0])])
        y = np.concatenate([v[sel].astype(np.float64), np.zeros(B.shape[0])])
        c = np.linalg.lstsq(M, y, rcond=None)[0]
        np.testing.assert_allclose(C[f], c, rtol=0, atol=2e-3 * np.abs(c).max())
        np.testing.assert_allclose(X[f], B.T @ c, rtol=0, atol=2e-3 * np.abs(B.T @ c).max() * 3)


# ------------------------------------------------------- P4 exact recovery
def test_exact_recovery_noiseless_low_rank(oracle_lib):
    """A noiseless rank-2 30 x 30 matrix with 60 % of cells observed is
    recovered by the full-gradient fit (lambda = 0): held-out RMSE < 1e-6."""
    R, u, i = synth.dense_lowrank_case(30, 30, 2, 0.6, seed=7)
    R = R.astype(np.float32).astype(np.float64)
    g = np.random.default_rng(1)
    ho = g.random(u.size) < 0.1
    a, b = u[~ho], i[~ho]
    P0 = g.normal(0, 0.3, (30, 2))
    Q0 = g.normal(0, 0.3, (30, 2))
    st, P, Q, h, _ = oracle_lib.fit(a, b, R[a, b].astype(np.float32), P0, Q0, 20000, 0.0, 0.5,
                                    "degree")
    assert st == 0
    pred = (P @ Q.T)[u[ho], i[ho]]
    rmse = float(np.sqrt(np.mean((pred - R[u[ho], i[ho]]) ** 2)))
    assert rmse < 1e-6


# ------------------------------------------------------- P5 monotone descent
@pytest.mark.parametrize("step,lr", [("sum", 0.02), ("degree", 0.15)])
def test_monotone_descent_small_step(oracle_lib, step, lr):
    """Full-gradient descent with a small step never increases Eq. 2 (the
    degree step is gradient descent preconditioned by a positive diagonal)."""
    p = synth.tiny()
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    st, P, Q, h, _ = oracle_lib.fit(a, b, v, p.P0, p.Q0, 200, p.lam, lr, step)
    assert st == 0
    assert np.all(np.diff(h) <= 0.0)
    assert h[-1] < 0.01 * h[0]


# ------------------------------------------------------- P7 TSID identity
def test_tsid_skeleton_identity(oracle_lib):
    """Theorem 1 (Section 3.1): for an exactly rank-k, fully observed R and
    |I| = |J| = k with a nonsingular core, W_L R*_k W_R^T = R_k.  Checked twice:
    (1) the theorem's own formula with U_1, V_1 from numpy's SVD; (2) the
    method's pipeline in the oracle -- fit the k x k template to zero loss,
    extend the free rows from the template columns, then every free column
    from all rows (lambda = 0, exact ridge solves) -- reproduces R."""
    k, m, n = 3, 12, 10
    g = np.random.default_rng(11)
    # integer factors: R is exactly rank k and exactly representable in fp32
    R = (g.integers(-3, 4, (m, k)) @ g.integers(-3, 4, (n, k)).T).astype(np.float64)
    I = np.array([1, 5, 8])
    J = np.array([0, 4, 7])
    assert np.linalg.matrix_rank(R) == k and abs(np.linalg.det(R[np.ix_(I, J)])) > 0.5
    U, S, Vt = np.linalg.svd(R)
    U1, V1 = U[:, :k], Vt[:k].T
    WL = U1 @ np.linalg.inv(U1[I])
    WR = V1 @ np.linalg.inv(V1[J])
    np.testing.assert_allclose(WL @ R[np.ix_(I, J)] @ WR.T, R, atol=1e-9)

    aa, bb = _full_cells(k, k)
    core = R[np.ix_(I, J)]
    g = np.random.default_rng(3)
    st, P, Q, h, _ = oracle_lib.fit(aa, bb, core[aa, bb].astype(np.float32), g.normal(0, .5, (k, k)),
                                    g.normal(0, .5, (k, k)), 20000, 0.0, 0.02, "sum")
    assert st == 0 and h[-1] < 1e-24
    free_rows = np.setdiff1d(np.arange(m), I)
    Qfull = np.zeros((n, k))
    Qfull[J] = Q
    fr, fc = np.meshgrid(np.arange(free_rows.size), J, indexing="ij")
    fr, fc = fr.ravel(), fc.ravel()
    st, Pfree = oracle_lib.ridge(fc, fr, R[free_rows[fr], fc].astype(np.float32), free_rows.size,
                                 Qfull, 0.0)
    assert st == 0
    Pfull = np.zeros((m, k))
    Pfull[I] = P
    Pfull[free_rows] = Pfree
    free_cols = np.setdiff1d(np.arange(n), J)
    rr, cc = np.meshgrid(np.arange(m), np.arange(free_cols.size), indexing="ij")
    rr, cc = rr.ravel(), cc.ravel()
    st, Qfree = oracle_lib.ridge(rr, cc, R[rr, free_cols[cc]].astype(np.float32), free_cols.size,
                                 Pfull, 0.0)
    assert st == 0
    Qfull[free_cols] = Qfree
    np.testing.assert_allclose(Pfull @ Qfull.T, R, atol=1e-6)


# ---------------------------------------------------------------- P8 clip
def test_clip_table_and_infinite_threshold(oracle_lib):
    """Section 5.3: min(max(xi, -g), g) == min(g, xi) per coordinate: values
    above xi become xi, the rest pass.  A one-cell problem (k = 1, lambda = 0,
    q = 1, p = 0) has descent direction d = 2 r for p, so r sets d."""
    xi = 0.1
    one = np.zeros(1, np.int32)
    for d in [-1.0, 0.0, xi / 2, xi, 2 * xi, 7.0]:
        st, P, Q, h, _ = oracle_lib.fit(one, one, np.array([d / 2], np.float32),
                                        np.array([[0.0]]), np.array([[1.0]]), 1, 0.0, 1.0, "sum",
                                        True, xi)
        assert st == 0
        want = min(float(np.float32(d / 2)) * 2, xi)
        assert P[0, 0] == want
    # xi = +inf reproduces the unclipped trajectory bit for bit
    p = synth.tiny()
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    r1 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 10, p.lam, p.lr, "sum", False)
    r2 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 10, p.lam, p.lr, "sum", True, math.inf)
    assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2])
    assert np.array_equal(r1[3], r2[3])


def test_nonfinite_stops_at_last_finite_iterate(oracle_lib):
    """A step size that overflows ends the fit with status 7; the factors are
    those of the last epoch whose update stayed finite."""
    p = synth.tiny()
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    st, P, Q, h, done = oracle_lib.fit(a, b, v, p.P0, p.Q0, 100, p.lam, 1e6, "sum")
    assert st == 7 and 0 < done < 100
    st2, P2, Q2, h2, _ = oracle_lib.fit(a, b, v, p.P0, p.Q0, done, p.lam, 1e6, "sum")
    assert st2 == 0 and np.array_equal(P, P2) and np.array_equal(Q, Q2)
    assert np.all(np.isfinite(P)) and np.array_equal(h[:done + 1], h2, equal_nan=True)


# ---------------------------------------------------------------- P9 bf16
def test_bf16_round_to_nearest_even_matches_torch(oracle_lib):
    """bf16 rounding of the factors (bf16 mode) is IEEE round-to-nearest-even,
    checked bit for bit against torch's float32 -> bfloat16 conversion."""
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(0)
    bits = g.integers(0, 2 ** 32, 20000, dtype=np.uint64).astype(np.uint32)
    ties = (g.integers(0, 2 ** 16, 2000, dtype=np.uint64).astype(np.uint32) << 16) | 0x8000
    special = np.array([0x00000000, 0x80000000, 0x7F800000, 0xFF800000, 0x7F7FFFFF, 0x00000001,
                        0x00008000, 0x00018000, 0x3F808000, 0x3F818000, 0x7F7F8000], np.uint32)
    allb = np.concatenate([bits, ties, special])
    f = allb.view(np.float32)
    ref = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    ours = np.array([oracle_lib.bf16_bits(float(x)) for x in f], np.uint16)
    nan = np.isnan(f)
    assert np.array_equal(ours[~nan], ref[~nan])
    ours_f = (ours[nan].astype(np.uint32) << 16).view(np.float32)
    assert np.all(np.isnan(ours_f))


def test_bf16_mode_fit_tracks_fp64(oracle_lib):
    """bf16 mode changes the products only by bf16 rounding (relative 2^-9):
    on Tiny its loss history stays within 1 % of the fp64 run."""
    p = synth.tiny()
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    h64 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 30, p.lam, 0.02, "sum")[3]
    h16 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 30, p.lam, 0.02, "sum", bf16=True)[3]
    np.testing.assert_allclose(h16, h64, rtol=1e-2)
    assert not np.array_equal(h16, h64)


# ------------------------------------------------------- P10 index work
def test_template_maps_filter_and_buckets_brute_force(oracle_lib):
    """Maps, Omega* and both bucket orders against Python dicts and sorted()."""
    p = synth.random_case(23, 17, 150, 9, 6, 4, seed=3)
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    assert st == 0
    pos_r = {int(u): a for a, u in enumerate(p.I)}
    pos_c = {int(i): b for b, i in enumerate(p.J)}
    assert [pos_r.get(u, -1) for u in range(p.m)] == rm.tolist()
    assert [pos_c.get(i, -1) for i in range(p.n)] == cm.tolist()
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    want = [(pos_r[int(u)], pos_c[int(i)], float(r)) for u, i, r in zip(p.u, p.i, p.r)
            if int(u) in pos_r and int(i) in pos_c]
    assert list(zip(a.tolist(), b.tolist(), v.astype(np.float64).tolist())) == want
    bk = oracle_lib.bucket(a, b, v, p.I.size, p.J.size)
    csr = sorted(want)
    assert bk["csr_col"].tolist() == [x[1] for x in csr]
    assert bk["csr_val"].astype(np.float64).tolist() == [x[2] for x in csr]
    csc = sorted(want, key=lambda x: (x[1], x[0]))
    assert bk["csc_row"].tolist() == [x[0] for x in csc]
    assert bk["csc_val"].astype(np.float64).tolist() == [x[2] for x in csc]
    for ptr, deg, key, n_ in ((bk["row_ptr"], bk["deg_r"], 0, p.I.size),
                              (bk["col_ptr"], bk["deg_c"], 1, p.J.size)):
        cnt = [sum(1 for x in want if x[key] == j) for j in range(n_)]
        assert deg.tolist() == cnt
        assert ptr[0] == 0 and ptr[-1] == len(want)
        assert np.all(np.diff(ptr) == deg)


def test_validation_codes(oracle_lib):
    """Out-of-range ids -> 2 (before duplicates), repeated ids / cells -> 3."""
    assert oracle_lib.template_maps(5, 4, [0, 5], [0])[0] == 2
    assert oracle_lib.template_maps(5, 4, [1, 1], [9])[0] == 2
    assert oracle_lib.template_maps(5, 4, [1, 1], [0])[0] == 3
    assert oracle_lib.template_maps(5, 4, [1, 2], [3, 3])[0] == 3
    assert oracle_lib.check_omega(3, 3, [0, 1], [0, 3], [1.0, 1.0]) == 2
    assert oracle_lib.check_omega(3, 3, [0, 1], [0, 1], [1.0, np.nan]) == 1
    assert oracle_lib.check_omega(3, 3, [0, 1, 0], [0, 1, 0], [1.0, 1.0, 2.0]) == 3
    assert oracle_lib.check_omega(3, 3, [0, 1, 2], [0, 1, 0], [1.0, 1.0, 2.0]) == 0


def test_chunk_plan_definition(oracle_lib):
    """Chunk boundaries against the definitions, computed another way
    (binary search on the prefix sums; an explicit greedy walk)."""
    g = np.random.default_rng(4)
    for trial in range(20):
        n_free = int(g.integers(0, 60))
        counts = g.integers(0, 50, n_free) * (g.random(n_free) < 0.8)
        if trial % 5 == 0 and n_free:
            counts[g.integers(0, n_free)] = 5000
        total = int(counts.sum())
        excl = np.concatenate([[0], np.cumsum(counts)])
        for K in (1, 3, 10):
            bnd = oracle_lib.chunk_plan(counts, n_chunks=K)
            want = [0] + [int(np.searchsorted(excl, -(-j * total // K), side="left"))
                          for j in range(1, K)] + [n_free]
            want = [min(x, n_free) for x in want]
            assert bnd.tolist() == want
        C = 120
        if trial == 0:  # an empty row ahead of one over the cap
            counts = np.array([0, 500, 20, 30])
            n_free = 4
        bnd = oracle_lib.chunk_plan(counts, max_entries=C).tolist()
        assert bnd[0] == 0 and bnd[-1] == n_free
        for s, e in zip(bnd[:-1], bnd[1:]):
            assert e > s
            tot = int(counts[s:e].sum())
            assert tot <= C or e - s == 1
            if e < n_free:
                assert tot + int(counts[e]) > C


# ------------------------------------------------------- NEXT-4 mini-batches
def test_splitmix64_published_outputs(oracle_lib):
    """The batch hash is SplitMix64's output function (Steele, Lea and Flood,
    2014): from state 0 the generator's first outputs are the published
    values, the state advancing by the golden-ratio increment."""
    gamma = 0x9E3779B97F4A7C15
    want = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]
    got = [oracle_lib.splitmix64((i * gamma) & (2 ** 64 - 1)) for i in range(4)]
    assert got == want


def test_minibatch_batches_are_balanced(oracle_lib):
    """Every cell falls in exactly one of B batches, and the batch sizes of
    many cells are those of a uniform draw (within five standard deviations)."""
    g = np.random.default_rng(4)
    a = g.integers(0, 5000, 40000)
    b = g.integers(0, 5000, 40000)
    for B in (2, 3, 8):
        idx = np.array([oracle_lib.batch_of(x, y, 11, B) for x, y in zip(a, b)])
        assert np.array_equal(oracle_lib.batch_of_many(a, b, 11, B), idx)
        assert idx.min() >= 0 and idx.max() < B
        cnt = np.bincount(idx, minlength=B)
        sd = math.sqrt(a.size * (1 / B) * (1 - 1 / B))
        assert np.all(np.abs(cnt - a.size / B) < 5 * sd), cnt


def _every_line_observed(seed, m, n, nnz):
    g = np.random.default_rng(seed)
    cells = {(x, int(g.integers(n))) for x in range(m)} | {(int(g.integers(m)), y) for y in range(n)}
    while len(cells) < nnz:
        cells.add((int(g.integers(m)), int(g.integers(n))))
    c = np.array(sorted(cells))
    return c[:, 0].astype(np.int32), c[:, 1].astype(np.int32), g.standard_normal(len(c)).astype(np.float32)


@pytest.mark.parametrize("step", ["sum", "degree"])
def test_minibatch_one_batch_is_the_full_gradient_epoch(oracle_lib, step):
    """With one batch every epoch is a single full-gradient step (Eqs. 3-5):
    the Jacobi fit's factors and losses, bit for bit, when every row and
    column has a cell (a line without one is left alone by a batch step)."""
    a, b, v = _every_line_observed(0, 30, 25, 300)
    g = np.random.default_rng(1)
    P0, Q0 = g.normal(0, .5, (30, 8)), g.normal(0, .5, (25, 8))
    r1 = oracle_lib.fit(a, b, v, P0, Q0, 6, 0.1, 0.01, step, True, 0.1)
    r2 = oracle_lib.fit_minibatch(a, b, v, P0, Q0, 6, 0.1, 0.01, step, True, 0.1, n_batches=1, seed=9)
    assert r1[0] == r2[0] == 0 and r2[4] == 6
    for x, y in zip(r1[1:4], r2[1:4]):
        assert np.array_equal(x, y)


def test_minibatch_two_batches_by_hand(oracle_lib):
    """One row and two columns, k = 1, each cell in its own batch (seed 2:
    cell (0, 0) in batch 0, cell (0, 1) in batch 1).  The first batch moves p
    and q0 by Eqs. 3-5 on its one cell and leaves q1 alone; the second moves p
    again, from its new value, and q1."""
    assert oracle_lib.batch_of(0, 0, 2, 2) == 0 and oracle_lib.batch_of(0, 1, 2, 2) == 1
    p, q0, q1, v0, v1, lam, lr = 0.7, -0.4, 1.3, 2.0, -1.0, 0.25, 0.1
    e = v0 - p * q0
    p1 = p - lr * (-2 * e * q0 + 2 * lam * p)
    q01 = q0 - lr * (-2 * e * p + 2 * lam * q0)
    e = v1 - p1 * q1
    p2 = p1 - lr * (-2 * e * q1 + 2 * lam * p1)
    q11 = q1 - lr * (-2 * e * p1 + 2 * lam * q1)
    loss0 = (v0 - p * q0) ** 2 + (v1 - p * q1) ** 2 + lam * (p * p + q0 * q0 + q1 * q1)
    for step in ("sum", "degree"):  # one cell per line per batch: both rules agree
        st, P, Q, h, done = oracle_lib.fit_minibatch(
            np.zeros(2, np.int32), np.array([0, 1], np.int32), np.array([v0, v1], np.float32),
            np.array([[p]]), np.array([[q0], [q1]]), 1, lam, lr, step, n_batches=2, seed=2)
        assert st == 0 and done == 1
        assert h[0] == pytest.approx(loss0, rel=1e-15)
        assert P[0, 0] == pytest.approx(p2, rel=1e-14)
        assert Q[0, 0] == pytest.approx(q01, rel=1e-14) and Q[1, 0] == pytest.approx(q11, rel=1e-14)


def test_minibatch_brute_force_tiny(oracle_lib):
    """Three batches on a tiny matrix against a per-cell Python sweep of the
    same rule: each batch's gradient from the factors the previous batch
    left, rows and columns divided by their cell count in the batch."""
    a, b, v = _every_line_observed(5, 6, 5, 18)
    g = np.random.default_rng(6)
    P0, Q0 = g.normal(0, .5, (6, 3)), g.normal(0, .5, (5, 3))
    lam, lr, B, seed, epochs = 0.2, 0.05, 3, 123, 3
    P, Q = P0.copy(), Q0.copy()
    for _ in range(epochs):
        for beta in range(B):
            gP, gQ = np.zeros_like(P), np.zeros_like(Q)
            dP, dQ = np.zeros(6), np.zeros(5)
            for x, y, r in zip(a, b, v):
                if oracle_lib.batch_of(x, y, seed, B) != beta:
                    continue
                err = float(r) - sum(P[x, c] * Q[y, c] for c in range(3))
                for c in range(3):
                    gP[x, c] -= 2 * err * Q[y, c]
                    gQ[y, c] -= 2 * err * P[x, c]
                dP[x] += 1
                dQ[y] += 1
            for F, G, D in ((P, gP, dP), (Q, gQ, dQ)):
                for x in range(F.shape[0]):
                    if D[x]:
                        F[x] = F[x] - lr * (G[x] + 2 * lam * F[x]) / D[x]
    st, Po, Qo, h, done = oracle_lib.fit_minibatch(a, b, v, P0, Q0, epochs, lam, lr, "degree",
                                                   n_batches=B, seed=seed)
    assert st == 0 and done == epochs
    np.testing.assert_allclose(Po, P, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(Qo, Q, rtol=1e-12, atol=1e-14)


def test_minibatch_nonfinite_reports_whole_epochs(oracle_lib):
    """A step size that overflows ends the mini-batch fit with status 7 and
    counts only the epochs that completed; the factors stay finite."""
    a, b, v = _every_line_observed(7, 20, 20, 150)
    g = np.random.default_rng(8)
    st, P, Q, h, done = oracle_lib.fit_minibatch(a, b, v, g.normal(0, 1, (20, 4)), g.normal(0, 1, (20, 4)),
                                                 100, 0.1, 1e6, "sum", n_batches=4, seed=1)
    assert st == 7 and 0 <= done < 100
    assert np.all(np.isfinite(P)) and np.all(np.isfinite(Q))


# ------------------------------------------ NEXT-4 per-entry clipping order
def test_per_entry_clip_without_regulariser_or_threshold_is_plain_descent(oracle_lib):
    """clip 2 with lambda = 0 and xi = inf adds each cell's 2 e q, whose sum is
    the negated data gradient exactly: the unclipped fit bit for bit (both
    step rules, Jacobi and mini-batch epochs)."""
    p = synth.tiny()
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    for step in ("sum", "degree"):
        lr = p.lr if step == "degree" else 0.01
        r0 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 5, 0.0, lr, step, 0, 0.1)
        r2 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 5, 0.0, lr, step, 2, math.inf)
        assert r0[0] == r2[0] == 0
        for x, y in zip(r0[1:4], r2[1:4]):
            assert np.array_equal(x, y)
        m0 = oracle_lib.fit_minibatch(a, b, v, p.P0, p.Q0, 3, 0.0, lr, step, 0, 0.1, n_batches=3, seed=4)
        m2 = oracle_lib.fit_minibatch(a, b, v, p.P0, p.Q0, 3, 0.0, lr, step, 2, math.inf, n_batches=3, seed=4)
        assert np.array_equal(m0[1], m2[1]) and np.array_equal(m0[2], m2[2])


def test_per_entry_clip_with_one_cell_per_line_is_the_summed_clip(oracle_lib):
    """A line with one cell has one term: clipping it before or after the
    sum is the same, bit for bit (cells on a permutation, both step rules)."""
    g = np.random.default_rng(3)
    n = 40
    a = np.arange(n, dtype=np.int32)
    b = g.permutation(n).astype(np.int32)
    v = g.normal(0, 2, n).astype(np.float32)
    P0, Q0 = g.normal(0, 1, (n, 4)), g.normal(0, 1, (n, 4))
    for step in ("sum", "degree"):
        r1 = oracle_lib.fit(a, b, v, P0, Q0, 6, 0.2, 0.05, step, 1, 0.05)
        r2 = oracle_lib.fit(a, b, v, P0, Q0, 6, 0.2, 0.05, step, 2, 0.05)
        for x, y in zip(r1[1:4], r2[1:4]):
            assert np.array_equal(x, y)


def test_per_entry_clip_by_hand(oracle_lib):
    """One row (p = 1) and two columns (q0 = 2, q1 = -1), values 5 and 0.5,
    lambda 0.1, xi 1, lr 0.1, sum step.  Residuals 3 and 1.5.  Per entry the
    row's terms are 11.8 -> 1 and -3.2, so p' = 1 + 0.1 (1 - 3.2) = 0.78; the
    summed direction would be 8.8 -> 1 and p' = 1.1.  Columns: 5.6 -> 1 and
    3.2 -> 1, so q0' = 2.1 and q1' = -0.9."""
    a = np.zeros(2, np.int32)
    b = np.array([0, 1], np.int32)
    v = np.array([5.0, 0.5], np.float32)
    P0, Q0 = np.array([[1.0]]), np.array([[2.0], [-1.0]])
    st, P, Q, h, _ = oracle_lib.fit(a, b, v, P0, Q0, 1, 0.1, 0.1, "sum", 2, 1.0)
    assert st == 0
    assert P[0, 0] == pytest.approx(0.78, rel=1e-14)
    assert Q[:, 0] == pytest.approx([2.1, -0.9], rel=1e-14)
    st, P, Q, h, _ = oracle_lib.fit(a, b, v, P0, Q0, 1, 0.1, 0.1, "sum", 1, 1.0)
    assert P[0, 0] == pytest.approx(1.1, rel=1e-14)


def test_per_entry_clip_brute_force_tiny(oracle_lib):
    """Two Jacobi epochs of the per-entry order against a per-cell Python
    sweep: every term from the same iterate, clipped, summed per line and
    divided by the line's cell count."""
    a, b, v = _every_line_observed(9, 7, 6, 20)
    g = np.random.default_rng(10)
    P0, Q0 = g.normal(0, .7, (7, 3)), g.normal(0, .7, (6, 3))
    lam, lr, xi = 0.3, 0.1, 0.2
    P, Q = P0.copy(), Q0.copy()
    dP, dQ = np.bincount(a, minlength=7), np.bincount(b, minlength=6)
    for _ in range(2):
        gP, gQ = np.zeros_like(P), np.zeros_like(Q)
        for x, y, r in zip(a, b, v):
            err = float(r) - sum(P[x, c] * Q[y, c] for c in range(3))
            for c in range(3):
                gP[x, c] += min(2 * err * Q[y, c] - 2 * lam * P[x, c], xi)
                gQ[y, c] += min(2 * err * P[x, c] - 2 * lam * Q[y, c], xi)
        P, Q = P + lr * gP / dP[:, None], Q + lr * gQ / dQ[:, None]
    st, Po, Qo, _, _ = oracle_lib.fit(a, b, v, P0, Q0, 2, lam, lr, "degree", 2, xi)
    assert st == 0
    np.testing.assert_allclose(Po, P, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(Qo, Q, rtol=1e-12, atol=1e-14)


def test_per_entry_clip_is_not_an_extension_option(oracle_lib):
    F = np.ones((3, 2))
    st, X = oracle_lib.extend(np.zeros(1, np.int32), np.zeros(1, np.int32), np.ones(1, np.float32), 1, F, 3,
                              0.1, 0.1, "degree", 2, 0.1)
    assert st == 1


# ------------------------------------------------ NEXT-4 multi-view term
def _sym_coo(S):
    """Off-diagonal nonzeros of a dense symmetric S as COO (both orientations)."""
    r, c = np.nonzero(S - np.diag(np.diag(S)))
    return r.astype(np.int32), c.astype(np.int32), S[r, c].astype(np.float32)


def test_similarity_from_attributes_brute_force(oracle_lib):
    """S_ii' = (1/J) sum_j [a_ij == a_i'j] (Section 2.2): a Python double loop,
    unit diagonal, symmetric."""
    g = np.random.default_rng(30)
    A = g.integers(0, 3, (9, 5))
    S = oracle_lib.similarity(A)
    want = np.array([[np.mean(A[i] == A[j]) for j in range(9)] for i in range(9)])
    assert np.array_equal(S, want) and np.all(np.diag(S) == 1.0) and np.array_equal(S, S.T)


def test_multiview_beta_zero_is_the_plain_fit(oracle_lib):
    p = synth.tiny()
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    S = oracle_lib.similarity(np.random.default_rng(31).integers(0, 4, (p.J.size, 3)))
    r, c, w = _sym_coo(S)
    r0 = oracle_lib.fit(a, b, v, p.P0, p.Q0, 5, p.lam, p.lr, "degree", True, 0.1)
    r1 = oracle_lib.fit_mv(a, b, v, p.P0, p.Q0, 5, p.lam, p.lr, r, c, w, 0.0, "degree", True, 0.1)
    for x, y in zip(r0[:4], r1[:4]):
        assert np.array_equal(x, y)


def test_multiview_gradient_matches_central_differences(oracle_lib):
    """The objective with the similarity term, (beta/2) sum S_ii' ||q_i - q_i'||^2,
    has the printed update term 2 beta sum_i' S_ii' (q_i - q_i') as its
    gradient: one epoch's step against central differences of the loss
    (quadratic per coordinate, so exact up to rounding)."""
    p = synth.random_case(9, 7, 30, 9, 7, 3, seed=21, lam=0.3)
    st, rm, cm = oracle_lib.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle_lib.filter_template(p.u, p.i, p.r, rm, cm)
    S = oracle_lib.similarity(np.random.default_rng(32).integers(0, 3, (7, 4)))
    r, c, w = _sym_coo(S)
    beta, lr = 0.7, 1e-3
    P0, Q0 = p.P0.astype(np.float64), p.Q0.astype(np.float64)
    st, P1, Q1, h, _ = oracle_lib.fit_mv(a, b, v, P0, Q0, 1, p.lam, lr, r, c, w, beta, "sum")
    assert st == 0
    h_ = 1e-3
    for X, G, isP in ((P0, (P0 - P1) / lr, True), (Q0, (Q0 - Q1) / lr, False)):
        for idx in np.ndindex(*X.shape):
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += h_
            Xm[idx] -= h_
            args = ((Xp, Q0), (Xm, Q0)) if isP else ((P0, Xp), (P0, Xm))
            Lp, Lm = (oracle_lib.loss_mv(a, b, v, 9, 7, PP, QQ, p.lam, r, c, w, beta) for PP, QQ in args)
            fd = (Lp - Lm) / (2 * h_)
            assert abs(fd - G[idx]) <= 1e-8 * max(1.0, abs(fd)), (isP, idx, fd, G[idx])
    direct = oracle_lib.loss(a, b, v, 9, 7, P0, Q0, p.lam) + beta / 2 * sum(
        S[i, j] * ((Q0[i] - Q0[j]) ** 2).sum() for i in range(7) for j in range(7))
    assert h[0] == pytest.approx(direct, rel=1e-13)


def test_multiview_without_cells_is_laplacian_smoothing(oracle_lib):
    """No observed cells and lambda = 0: one epoch is Q <- Q - 2 lr beta (D - S) Q
    with D the diagonal of S's row sums (the graph Laplacian), P unchanged."""
    g = np.random.default_rng(33)
    S = oracle_lib.similarity(g.integers(0, 3, (8, 4)))
    r, c, w = _sym_coo(S)
    Sf = np.zeros((8, 8))
    Sf[r, c] = w.astype(np.float64)
    Lap = np.diag(Sf.sum(1)) - Sf
    P0, Q0 = g.normal(0, 1, (5, 3)), g.normal(0, 1, (8, 3))
    beta, lr = 0.4, 0.05
    none = np.zeros(0, np.int32)
    st, P1, Q1, _, _ = oracle_lib.fit_mv(none, none, np.zeros(0, np.float32), P0, Q0, 1, 0.0, lr, r, c, w, beta)
    assert st == 0 and np.array_equal(P1, P0)
    np.testing.assert_allclose(Q1, Q0 - 2 * lr * beta * Lap @ Q0, rtol=1e-13, atol=1e-15)


def test_multiview_rejections(oracle_lib):
    none = np.zeros(0, np.int32)
    P0, Q0 = np.ones((2, 2)), np.ones((3, 2))
    bad = (np.array([0], np.int32), np.array([3], np.int32), np.ones(1, np.float32))
    assert oracle_lib.fit_mv(none, none, np.zeros(0, np.float32), P0, Q0, 1, 0.1, 0.1, *bad, 0.5)[0] == 2
    ok = (np.array([0, 1], np.int32), np.array([1, 0], np.int32), np.ones(2, np.float32))
    assert oracle_lib.fit_mv(none, none, np.zeros(0, np.float32), P0, Q0, 1, 0.1, 0.1, *ok, 0.5, "sum", 2,
                             0.1)[0] == 1
