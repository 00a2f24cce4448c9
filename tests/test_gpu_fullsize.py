"""Parity at full benchmark size, in the launch configuration bench.py times.

Sampled: one full-gradient epoch from (P0, Q0): the new row p_a depends
only on the cells of row a and on Q0, so the oracle, given just the cells of
a sample of rows (or columns), reproduces those rows exactly.  The loss
L(P0, Q0) over all of Omega* is checked as a whole.

Whole fits: several epochs over every cell of the template against the
oracle's line-parallel fit (or_fit_lines built with OpenMP, the same bits as
the serial oracle): Scientific (fp32) 5 epochs, every factor within 1e-4
relative Frobenius error; Rating-shaped (bf16) its 20 epochs and
Billion-scale (bf16) 5 epochs, held-out RMSE within 1e-2 relative.
"""
import functools
import math
import time

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import gpu_fit, note, oracle_template, rel_fro

pytestmark = pytest.mark.gpu


@functools.lru_cache(maxsize=None)
def _problem(name):
    note(f"fullsize: generating {name}")
    t0 = time.perf_counter()
    p = synth.make(name)
    note(f"fullsize: {name} has {p.nnz} training cells ({time.perf_counter() - t0:.0f}s)")
    return p


def _sampled_parity(T, p, n_rows=64, n_cols=64, tol=1e-4):
    rm, cm, a, b, v = oracle_template(p)
    note(f"fullsize {p.name}: building template over {p.nnz} cells")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    assert T.info()["nnz"] == a.size
    st, P1, Q1, hist = gpu_fit(T, p, epochs=1)
    assert st == 0
    g = np.random.default_rng(0)
    # a uniform sample plus the four longest buckets of each side (those span
    # several waves, so their updates go through the fixup kernel)
    top_r = np.argsort(-np.bincount(a, minlength=p.I.size), kind="stable")[:4]
    top_c = np.argsort(-np.bincount(b, minlength=p.J.size), kind="stable")[:4]
    rows = np.union1d(g.choice(p.I.size, n_rows, replace=False), top_r)
    cols = np.union1d(g.choice(p.J.size, n_cols, replace=False), top_c)
    bf16 = p.prec == "bf16"
    if bf16:
        # the automatic rule takes the dense head tiles (16 x 16 tiles holding
        # at least ceil(fill * 256) cells, fill 0.15, or 0.10 at k = 128: 39
        # or 26 cells) when they hold a tenth of the cells: the library's
        # count must equal one made here, and rows of stripes with tiles join
        # the sample
        thr = math.ceil((0.10 if p.k >= 128 else 0.15) * 256)
        n_ti, n_tj = (p.I.size + 15) // 16, (p.J.size + 15) // 16
        cnt = np.bincount((a // 16).astype(np.int64) * n_tj + b // 16, minlength=n_ti * n_tj)
        dense = (cnt >= thr).reshape(n_ti, n_tj)
        cells = int(cnt[cnt >= thr].sum())
        del cnt
        info = T.dense_info()
        if cells >= 0.10 * a.size:
            assert info["cells"] == cells and info["tiles"] == int(dense.sum())
            sr = np.flatnonzero(dense.any(axis=1))
            sc = np.flatnonzero(dense.any(axis=0))
            rows = np.union1d(rows, np.minimum(g.choice(sr, 16) * 16 + g.integers(0, 16, 16), p.I.size - 1))
            cols = np.union1d(cols, np.minimum(g.choice(sc, 16) * 16 + g.integers(0, 16, 16), p.J.size - 1))
        else:
            assert info["tiles"] == 0
        del dense
    mask = np.zeros(p.I.size, dtype=bool)
    mask[rows] = True
    sel = mask[a]
    _, Po, _, _, _ = oracle.fit(a[sel], b[sel], v[sel], p.P0, p.Q0, 1, p.lam, p.lr, p.step, p.clip,
                                p.xi, bf16=bf16)
    assert rel_fro(P1[rows], Po[rows]) <= tol
    mask = np.zeros(p.J.size, dtype=bool)
    mask[cols] = True
    sel = mask[b]
    _, _, Qo, _, _ = oracle.fit(a[sel], b[sel], v[sel], p.P0, p.Q0, 1, p.lam, p.lr, p.step, p.clip,
                                p.xi, bf16=bf16)
    assert rel_fro(Q1[cols], Qo[cols]) <= tol
    if not bf16:
        L0 = oracle.loss(a, b, v, p.I.size, p.J.size, p.P0, p.Q0, p.lam)
        assert abs(hist[0] - L0) <= 1e-6 * L0


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    yield t
    t.close()


@pytest.mark.timeout(300)
def test_scientific_fullsize_sampled(T):
    _sampled_parity(T, _problem("scientific"))


@pytest.mark.timeout(400)
def test_rating_fullsize_sampled_bf16(T):
    _sampled_parity(T, _problem("rating"))


@pytest.mark.timeout(900)
def test_billion_fullsize_sampled_bf16(T):
    """1,000,000 x 100,000 template, about 4.2e8 training cells, k = 128."""
    _sampled_parity(T, _problem("billion"))


def _batch_ptr(own, rows, beta, B):
    cnt = np.bincount(beta.astype(np.int64) * rows + own, minlength=B * rows)
    return np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)


@pytest.mark.timeout(400)
def test_rating_fullsize_minibatch(T):
    """Mini-batch epochs at full size (bench.py --config rating --minibatch 8,
    seed 1).  A batch step depends on the factors every earlier step left, so
    no row of a later batch can be recomputed from its own cells; instead:
    the batch pointers of both sides bit-exact against the oracle's batch
    rule over all 38.8 M cells, and with one batch the epochs equal the Jacobi
    item-pass epochs bit for bit on every line with a cell (same plans, same
    stream order) while lines without one keep their start rows."""
    p = _problem("rating")
    rm, cm, a, b, v = oracle_template(p)
    note(f"fullsize minibatch rating: building template over {p.nnz} cells")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    try:
        T.set_minibatch(8, 1)
        st, P8, Q8, h8 = gpu_fit(T, p, epochs=1)
        assert st == 0 and np.all(np.isfinite(P8)) and np.all(np.isfinite(h8))
        beta = oracle.batch_of_many(a, b, 1, 8)
        assert np.array_equal(T.export_index("batch_ptr_r"), _batch_ptr(a, p.I.size, beta, 8))
        assert np.array_equal(T.export_index("batch_ptr_c"), _batch_ptr(b, p.J.size, beta, 8))
        del beta
        T.set_dense_tiles(0)
        T.set_pass_kernel("item")
        T.set_minibatch(1, 1)
        note("fullsize minibatch rating: one batch against the Jacobi epochs")
        st1, P1, Q1, h1 = gpu_fit(T, p, epochs=2)
        T.set_minibatch(0)
        stj, Pj, Qj, hj = gpu_fit(T, p, epochs=2)
    finally:
        T.set_minibatch(0)
        T.set_dense_tiles(-1)
        T.set_pass_kernel("auto")
    assert st1 == stj == 0
    dr = np.bincount(a, minlength=p.I.size) > 0
    dc = np.bincount(b, minlength=p.J.size) > 0
    assert np.array_equal(P1[dr], Pj[dr]) and np.array_equal(Q1[dc], Qj[dc])
    assert np.array_equal(P1[~dr], p.P0[~dr].astype(np.float32))
    assert np.array_equal(Q1[~dc], p.Q0[~dc].astype(np.float32))
    np.testing.assert_allclose(h1, hj, rtol=1e-6)


@pytest.mark.timeout(400)
def test_scientific_fullsize_variants_sampled(T):
    """The per-entry clip (bench.py --clip-per-entry) and the multi-view term
    (bench.py --similarity 0.01) at full Scientific size, one epoch from
    (P0, Q0): a row's new p depends only on its own cells and Q0, a column's
    new q on its cells, P0 and (with the term) its neighbours' rows of Q0, so
    the oracle reproduces sampled rows and columns from those alone."""
    import torch
    from paper_2608_00977_amd import make_opts
    p = _problem("scientific")
    rm, cm, a, b, v = oracle_template(p)
    note(f"fullsize scientific variants: building template over {p.nnz} cells")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    g = np.random.default_rng(1)
    rows = np.sort(g.choice(p.I.size, 48, replace=False))
    cols = np.sort(g.choice(p.J.size, 48, replace=False))
    sr, sc, sv = synth.similarity_graph(p.J.size, 16, 7)
    for variant in ("per_entry", "similarity"):
        clip = "per_entry" if variant == "per_entry" else p.clip
        beta = 0.01 if variant == "similarity" else 0.0
        T.set_similarity(sr, sc, sv, beta)
        P = torch.from_numpy(np.ascontiguousarray(p.P0, np.float32)).cuda()
        Q = torch.from_numpy(np.ascontiguousarray(p.Q0, np.float32)).cuda()
        note(f"fullsize scientific {variant}: one epoch")
        st, _ = T.fit_template(P, Q, make_opts(epochs=1, lam=p.lam, lr=p.lr, clip=clip, xi=p.xi, prec="fp32",
                                               step=p.step), raise_on_error=False)
        assert st == 0
        P1, Q1 = P.cpu().numpy(), Q.cpu().numpy()
        mr = np.zeros(p.I.size, bool)
        mr[rows] = True
        mc = np.zeros(p.J.size, bool)
        mc[cols] = True
        for mask, sel_of, out, idx in ((mr, a, P1, rows), (mc, b, Q1, cols)):
            sel = mask[sel_of]
            if variant == "per_entry":
                _, Po, Qo, _, _ = oracle.fit(a[sel], b[sel], v[sel], p.P0, p.Q0, 1, p.lam, p.lr, p.step, 2, p.xi)
            else:
                _, Po, Qo, _, _ = oracle.fit_mv(a[sel], b[sel], v[sel], p.P0, p.Q0, 1, p.lam, p.lr, sr, sc, sv, beta,
                                                p.step, p.clip, p.xi)
            ref = Po if out is P1 else Qo
            assert rel_fro(out[idx], ref[idx]) <= 1e-4, (variant, rel_fro(out[idx], ref[idx]))
    T.set_similarity(sr, sc, sv, 0.0)


def _oracle_fit_lines(a, b, v, p, epochs, per_call, bf16):
    """The OpenMP oracle over all cells, a few epochs per call (the state
    between calls is the fp64 factors, so the bits equal one long call)."""
    P, Q = p.P0, p.Q0
    hist = []
    done = 0
    while done < epochs:
        ep = min(per_call, epochs - done)
        t0 = time.perf_counter()
        st, P, Q, h, _ = oracle.fit_lines(a, b, v, P, Q, ep, p.lam, p.lr, p.step, p.clip, p.xi, bf16=bf16)
        assert st == 0
        hist.extend(h[:-1] if done + ep < epochs else h)
        done += ep
        note(f"fullsize oracle: {done}/{epochs} epochs on {oracle.threads()} threads "
             f"({time.perf_counter() - t0:.0f}s)")
    return P, Q, np.array(hist)


def _heldout_rmse_gpu(p, P, Q):
    import torch
    import paper_2608_00977_amd as tsid
    Tt = tsid.Tsid(0)
    try:
        Tt.build_template(p.m, p.n, p.tu, p.ti, p.tr, p.I, p.J, p.k)
        n_test = Tt.info()["nnz"]
        sse = Tt.loss(torch.from_numpy(np.ascontiguousarray(P, np.float32)).cuda(),
                      torch.from_numpy(np.ascontiguousarray(Q, np.float32)).cuda(), 0.0)
    finally:
        Tt.close()
    return float(np.sqrt(sse / max(1, n_test))), n_test


def _heldout_rmse_oracle(p, P, Q):
    st, rm, cm = oracle.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle.filter_template(p.tu, p.ti, p.tr, rm, cm)
    st, _, _, h, _ = oracle.fit_lines(a, b, v, P, Q, 0, 0.0, 1.0, "sum", False, 1.0)
    return float(np.sqrt(h[0] / max(1, a.size))), a.size


@pytest.mark.timeout(400)
def test_scientific_fullsize_five_epochs(T):
    """Scientific (fp32, k = 32, the slab pass): 5 epochs over all 24 M
    training cells; every row of P and Q within 1e-4 of the oracle."""
    p = _problem("scientific")
    rm, cm, a, b, v = oracle_template(p)
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    st, P, Q, hist = gpu_fit(T, p, epochs=5)
    assert st == 0
    note(f"fullsize scientific five epochs: pass kernels {T.pass_kernels()}")
    Po, Qo, ho = _oracle_fit_lines(a, b, v, p, 5, 5, False)
    eP, eQ = rel_fro(P, Po), rel_fro(Q, Qo)
    note(f"fullsize scientific: rel err P {eP:.2e} Q {eQ:.2e}")
    assert eP <= 1e-4 and eQ <= 1e-4
    np.testing.assert_allclose(hist, ho, rtol=1e-3)
    assert abs(hist[0] - ho[0]) <= 1e-6 * ho[0]


@pytest.mark.timeout(600)
def test_rating_fullsize_heldout_rmse_bf16(T):
    """Rating-shaped (bf16, k = 64, clip, dense tiles by the automatic rule):
    the benchmark's 20 epochs over all 38.8 M training cells; held-out RMSE
    within 1e-2 relative of the oracle's bf16 mode, and the training loss
    history within 1e-2."""
    p = _problem("rating")
    rm, cm, a, b, v = oracle_template(p)
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    st, P, Q, hist = gpu_fit(T, p, epochs=p.epochs)
    assert st == 0
    Po, Qo, ho = _oracle_fit_lines(a, b, v, p, p.epochs, 10, True)
    rg, n_test = _heldout_rmse_gpu(p, P, Q)
    ro, n_test_o = _heldout_rmse_oracle(p, Po, Qo)
    note(f"fullsize rating: held-out RMSE gpu {rg:.6f} oracle {ro:.6f} over {n_test} cells; "
         f"factor rel err P {rel_fro(P, Po):.2e} Q {rel_fro(Q, Qo):.2e}")
    assert n_test == n_test_o
    assert abs(rg - ro) <= 1e-2 * ro
    np.testing.assert_allclose(hist, ho, rtol=1e-2)


@pytest.mark.timeout(900)
def test_billion_fullsize_five_epochs_bf16(T):
    """Billion-scale (bf16, k = 128, clip, dense tiles and row-blocked Q
    passes by the automatic rules): 5 epochs over all 4.2e8 training cells;
    held-out RMSE (4.7e7 cells) within 1e-2 relative of the OpenMP oracle's
    bf16 mode, and the training loss history within 1e-2."""
    p = _problem("billion")
    rm, cm, a, b, v = oracle_template(p)
    del rm, cm
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    st, P, Q, hist = gpu_fit(T, p, epochs=5)
    assert st == 0
    note(f"fullsize billion: gpu fit done, row blocks {T.row_blocks()}, dense {T.dense_info()}")
    Po, Qo, ho = _oracle_fit_lines(a, b, v, p, 5, 2, True)
    del a, b, v
    rg, n_test = _heldout_rmse_gpu(p, P, Q)
    ro, n_test_o = _heldout_rmse_oracle(p, Po, Qo)
    note(f"fullsize billion: held-out RMSE gpu {rg:.6f} oracle {ro:.6f} over {n_test} cells; "
         f"factor rel err P {rel_fro(P, Po):.2e} Q {rel_fro(Q, Qo):.2e}")
    assert n_test == n_test_o
    assert abs(rg - ro) <= 1e-2 * ro
    np.testing.assert_allclose(hist, ho, rtol=1e-2)
