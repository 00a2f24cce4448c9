"""The multi-view similarity term (tsid_set_similarity; the item update of
Section 5.1 with the similarity matrix of Eq. 1) against the oracle's fit_mv,
through the C ABI.

S comes from seeded categorical attributes by the similarity of Section 2.2
(the oracle's `similarity`), kept where at least three of four attributes
agree.  Bars: those of the full-gradient fit (fp32 factors within 1e-4
relative Frobenius error, loss trajectory within 1e-3, final loss within
1e-6 of the oracle's extended loss at the library's own factors; bf16
held-out RMSE within 1e-2); with no observed cells one epoch is Laplacian
smoothing, checked against numpy within fp32 rounding.
"""
import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, oracle_rmse, oracle_template, rel_fro

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
LOSS_KERNEL_TOL = 1e-6
LOSS_TRAJ_TOL = 1e-3
BF16_RMSE_TOL = 1e-2


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    yield t
    t.close()


def _sim(n, seed, keep=0.75):
    """Sparse symmetric S over n columns (COO, both orientations, no diagonal)."""
    A = np.random.default_rng(seed).integers(0, 3, (n, 4))
    S = oracle.similarity(A)
    np.fill_diagonal(S, 0.0)
    r, c = np.nonzero(S >= keep)
    return r.astype(np.int32), c.astype(np.int32), S[r, c].astype(np.float32)


def _case(name):
    if name == "ragged_k32":
        return synth.random_case(700, 500, 9000, 300, 200, 32, seed=11, hot_rows=3, hot_cols=2, epochs=6,
                                 step="degree", lr=0.1, clip=True, xi=0.05), 0.05
    if name == "ragged_k8_sum":
        return synth.random_case(333, 257, 4000, 101, 77, 8, seed=12, hot_rows=1, epochs=5, step="sum",
                                 lr=0.02), 0.02
    if name == "ragged_k128":
        return synth.random_case(300, 280, 6000, 160, 140, 128, seed=15, hot_rows=1, hot_cols=1, epochs=3,
                                 step="degree", lr=0.1), 0.1
    if name == "sparse_empty":  # columns without cells move by the similarity term alone
        return synth.random_case(2000, 1500, 600, 700, 500, 32, seed=16, epochs=4, step="degree", lr=0.05), 0.1
    raise KeyError(name)


def _fit(T, p, prec="fp32", epochs=None, clip=None, lr=None):
    import torch
    from paper_2608_00977_amd import make_opts
    P = torch.from_numpy(np.ascontiguousarray(p.P0, np.float32)).cuda()
    Q = torch.from_numpy(np.ascontiguousarray(p.Q0, np.float32)).cuda()
    opts = make_opts(epochs=p.epochs if epochs is None else epochs, lam=p.lam, lr=p.lr if lr is None else lr,
                     clip=p.clip if clip is None else clip, xi=p.xi, prec=prec, step=p.step)
    st, hist = T.fit_template(P, Q, opts, raise_on_error=False)
    return st, P.cpu().numpy(), Q.cpu().numpy(), hist


@pytest.mark.parametrize("name", ["ragged_k32", "ragged_k8_sum", "ragged_k128", "sparse_empty"])
def test_multiview_fit_matches_oracle(T, name):
    p, beta = _case(name)
    r, c, w = _sim(p.J.size, 40)
    note(f"multiview {name} k={p.k} |S|={w.size} beta={beta}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_similarity(r, c, w, beta)
    st, P, Q, hist = _fit(T, p)
    assert st == 0 and T.pass_kernels() == ("item", "item")
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit_mv(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, r, c, w, beta, p.step,
                                       p.clip, p.xi)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL, rel_fro(P, Po)
    assert rel_fro(Q, Qo) <= FP32_TOL, rel_fro(Q, Qo)
    at_gpu = oracle.loss_mv(a, b, v, p.I.size, p.J.size, P, Q, p.lam, r, c, w, beta)
    assert abs(hist[-1] - at_gpu) <= LOSS_KERNEL_TOL * at_gpu
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)
    # the term matters here: without it the oracle ends elsewhere
    _, Pn, Qn, _, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, p.clip, p.xi)
    assert rel_fro(Qo, Qn) > 10 * FP32_TOL


def test_multiview_without_cells_is_laplacian_smoothing(T):
    """A template that holds no observed cell and lambda = 0: one epoch moves
    Q by -2 lr beta (D - S) Q (numpy, fp64) and leaves P alone."""
    import torch
    from paper_2608_00977_amd import make_opts
    k, n_t, beta, lr = 16, 96, 0.3, 0.05
    r, c, w = _sim(n_t, 41)
    g = np.random.default_rng(42)
    P0 = g.normal(0, 1, (10, k)).astype(np.float32)
    Q0 = g.normal(0, 1, (n_t, k)).astype(np.float32)
    none = np.zeros(0, np.int32)
    T.build_template(20, 200, none, none, np.zeros(0, np.float32), np.arange(10, dtype=np.int32),
                     np.arange(n_t, dtype=np.int32), k)
    T.set_similarity(r, c, w, beta)
    note("multiview laplacian smoothing")
    P, Q = torch.from_numpy(P0).cuda(), torch.from_numpy(Q0).cuda()
    st, hist = T.fit_template(P, Q, make_opts(epochs=1, lam=0.0, lr=lr), raise_on_error=False)
    assert st == 0
    Sf = np.zeros((n_t, n_t))
    Sf[r, c] = w.astype(np.float64)
    Lap = np.diag(Sf.sum(1)) - Sf
    Q0d = Q0.astype(np.float64)
    want = Q0d - 2 * lr * beta * Lap @ Q0d
    assert np.array_equal(P.cpu().numpy(), P0)
    assert rel_fro(Q.cpu().numpy(), want) <= 1e-6
    term = beta / 2 * sum(Sf[i, j] * ((Q0d[i] - Q0d[j]) ** 2).sum() for i, j in zip(r, c))
    assert hist[0] == pytest.approx(term, rel=1e-6)


def test_multiview_bf16_with_dense_tiles(T):
    """bf16 with the automatic dense tiles: the item pass adds the similarity
    sums next to the tile sums; held-out RMSE within 1e-2 of the oracle's."""
    p = synth.mid()
    p.clip, p.lr = True, 0.05
    beta = 0.05
    r, c, w = _sim(p.J.size, 43, keep=1.0)
    note(f"multiview bf16 mid |S|={w.size}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_similarity(r, c, w, beta)
    st, P, Q, _ = _fit(T, p, prec="bf16", clip=True)
    assert st == 0 and T.dense_info()["tiles"] > 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, _, _ = oracle.fit_mv(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, r, c, w, beta, p.step, True,
                                      p.xi, bf16=True)
    assert sto == 0
    r_gpu, _ = oracle_rmse(P.astype(np.float64), Q.astype(np.float64), p)
    r_or, _ = oracle_rmse(Po, Qo, p)
    assert abs(r_gpu - r_or) <= BF16_RMSE_TOL * r_or, (r_gpu, r_or)


def test_multiview_off_and_rebuild_restore_the_plain_fit(T):
    p, beta = _case("ragged_k32")
    r, c, w = _sim(p.J.size, 44)
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_pass_kernel("item")
    try:
        note("multiview off")
        base = _fit(T, p)
        T.set_similarity(r, c, w, beta)
        on = _fit(T, p)
        T.set_similarity(r, c, w, 0.0)
        off = _fit(T, p)
        T.set_similarity(r, c, w, beta)
        T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)  # a new template has no S
        rebuilt = _fit(T, p)
    finally:
        T.set_pass_kernel("auto")
    assert not np.array_equal(on[2], base[2])
    for x in (off, rebuilt):
        assert np.array_equal(x[1], base[1]) and np.array_equal(x[2], base[2])
        assert np.array_equal(x[3], base[3])


def test_multiview_rejections(T):
    import paper_2608_00977_amd as tsid
    p, beta = _case("ragged_k8_sum")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    n = p.J.size
    E = tsid.binding

    def status(fn):
        try:
            fn()
        except tsid.TsidError as e:
            return e.status
        return E.OK

    two = np.array([0, 1], np.int32), np.array([1, 0], np.int32)
    assert status(lambda: T.set_similarity(*two, np.array([1.0, 0.5], np.float32), 0.1)) == E.E_INVAL
    assert status(lambda: T.set_similarity(*two, np.array([-1.0, -1.0], np.float32), 0.1)) == E.E_INVAL
    assert status(lambda: T.set_similarity(*two, np.ones(2, np.float32), -0.1)) == E.E_INVAL
    assert status(lambda: T.set_similarity(np.array([0, n], np.int32), np.array([n, 0], np.int32),
                                           np.ones(2, np.float32), 0.1)) == E.E_RANGE
    assert status(lambda: T.set_similarity(np.array([0, 1, 0], np.int32), np.array([1, 0, 1], np.int32),
                                           np.ones(3, np.float32), 0.1)) == E.E_DUP
    T.set_similarity(*two, np.ones(2, np.float32), 0.1)
    try:
        note("multiview rejected modes")
        T.set_pass_kernel("slab")
        assert _fit(T, p, epochs=1)[0] == E.E_INVAL
        T.set_pass_kernel("auto")
        assert _fit(T, p, epochs=1, clip="per_entry")[0] == E.E_INVAL
        T.set_minibatch(2, 1)
        assert _fit(T, p, epochs=1)[0] == E.E_INVAL
        T.set_minibatch(0)
        assert _fit(T, p, epochs=1)[0] == E.OK
    finally:
        T.set_pass_kernel("auto")
        T.set_minibatch(0)
        T.set_similarity(*two, np.ones(2, np.float32), 0.0)
