"""Parity of the dense head tiles with the fp64 oracle, through the C ABI.

With dense tiles on, the bf16 fit computes the gradient sums of Eqs. 3-4 for
the cells of 16 x 16 tiles that are at least `fill` full on the matrix cores
(bf16 factor copies, fp32 accumulation, the residual split into a bf16 high
part and a bf16 remainder) and the item pass adds them to the sums of the
other cells before the update of Eq. 5.  The epochs are those of the oracle's
bf16 mode (products of bf16-rounded factors, Section 5.3).

Bars:
- one epoch from the same start: P_1 and Q_1 within 1e-4 relative Frobenius
  error of the oracle's (both sides round the same fp32 P_0, Q_0 to bf16, so
  the only differences are the fp32 accumulation order and the residual's
  two-part split, about 2^-17 relative per term), and L(P_0, Q_0) within
  1e-5 relative (per-stripe and per-item fp32 sums of e^2);
- several epochs: the loss trajectory within 1e-2 relative (from the second
  epoch on, a bf16 copy can differ in its last bit where the fp32 and fp64
  masters straddle a rounding boundary) and held-out RMSE within 1e-2, the
  bar of every bf16 fit;
- bitwise repeatable, and 5 + 5 epochs equal 10.
"""
import math

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import gpu_fit, note, oracle_rmse, oracle_template, rel_fro, rmse_on

pytestmark = pytest.mark.gpu

EPOCH_TOL = 1e-4
LOSS0_TOL = 1e-5
LOSS_TRAJ_TOL = 1e-2
BF16_RMSE_TOL = 1e-2


def auto_fill(k):
    """The automatic rule's tile fill (tsid_set_dense_tiles): 0.15, and 0.10
    at k = 128."""
    return 0.10 if k >= 128 else 0.15


def _case(name):
    if name == "half_k32":  # density 1/2, fill 1/2: about half the tiles dense; ragged edges
        p = synth.random_case(400, 300, 60000, 250, 190, 32, seed=31, hot_rows=2, hot_cols=1,
                              epochs=1, step="degree", lr=0.2, prec="bf16")
        return p, 0.5
    if name == "half_k16_sum":
        p = synth.random_case(300, 260, 39000, 170, 201, 16, seed=32, epochs=1, step="sum",
                              lr=0.002, prec="bf16")
        return p, 0.5
    if name == "half_k64_clip":
        p = synth.random_case(350, 330, 57000, 211, 177, 64, seed=33, hot_cols=2, epochs=1,
                              step="degree", lr=0.2, prec="bf16", clip=True, xi=0.05)
        return p, 0.5
    if name == "half_k128":
        p = synth.random_case(260, 250, 32000, 150, 140, 128, seed=34, hot_rows=1, epochs=1,
                              step="degree", lr=0.2, prec="bf16")
        return p, 0.5
    if name == "all_dense_k32":  # every cell observed: every tile dense, no other cells
        p = synth.random_case(200, 180, 36000, 160, 144, 32, seed=35, epochs=1, step="degree",
                              lr=0.2, prec="bf16")
        return p, 0.25
    if name == "wide_k64":  # row stripes of about 30 dense tiles: split over two waves each
        p = synth.random_case(300, 1200, 180000, 100, 1000, 64, seed=38, epochs=1, step="degree",
                              lr=0.2, prec="bf16")
        return p, 0.5
    if name == "mid_zipf":  # Zipf head: the tiles of the most-observed rows and columns
        p = synth.mid()
        p.epochs, p.prec = 1, "bf16"
        return p, 0.25
    raise KeyError(name)


ONE_EPOCH = ["half_k32", "half_k16_sum", "half_k64_clip", "half_k128", "all_dense_k32", "wide_k64",
             "mid_zipf"]


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    yield t
    t.close()


def _build(T, p):
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)


def _tile_info(a, b, m_t, n_t, fill):
    """Tiles holding at least ceil(fill * 256) cells, their cells and the
    stripes of each side holding one (counted here from the oracle's
    template, independently of the library's build)."""
    n_ti, n_tj = (m_t + 15) // 16, (n_t + 15) // 16
    t = (a // 16).astype(np.int64) * n_tj + b // 16
    cnt = np.bincount(t, minlength=n_ti * n_tj).reshape(n_ti, n_tj)
    dense = cnt >= max(1, math.ceil(fill * 256))
    return dict(cells=int(cnt[dense].sum()), tiles=int(dense.sum()),
                stripes=[int(dense.any(axis=1).sum()), int(dense.any(axis=0).sum())])


@pytest.mark.parametrize("name", ONE_EPOCH)
def test_dense_one_epoch_matches_oracle(T, name):
    p, fill = _case(name)
    note(f"dense one epoch {name} k={p.k} nnz={p.nnz} m_t={p.I.size} n_t={p.J.size} fill={fill}")
    _build(T, p)
    T.set_dense_tiles(fill)
    try:
        st, P, Q, hist = gpu_fit(T, p, epochs=1, prec="bf16")
        info = T.dense_info()
    finally:
        T.set_dense_tiles(-1)
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    assert info == _tile_info(a, b, p.I.size, p.J.size, fill)
    assert info["tiles"] > 0
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, 1, p.lam, p.lr, p.step, p.clip, p.xi,
                                    bf16=True)
    assert sto == 0
    assert rel_fro(P, Po) <= EPOCH_TOL, rel_fro(P, Po)
    assert rel_fro(Q, Qo) <= EPOCH_TOL, rel_fro(Q, Qo)
    assert abs(hist[0] - ho[0]) <= LOSS0_TOL * ho[0], (hist[0], ho[0])


def test_dense_and_item_paths_agree(T):
    """The same epoch with the tiles off and on: both within the oracle bar."""
    p, fill = _case("half_k32")
    _build(T, p)
    note("dense vs item")
    T.set_dense_tiles(0)
    off = gpu_fit(T, p, epochs=1, prec="bf16")
    assert T.dense_info()["tiles"] == 0
    T.set_dense_tiles(fill)
    try:
        on = gpu_fit(T, p, epochs=1, prec="bf16")
    finally:
        T.set_dense_tiles(-1)
    assert off[0] == 0 and on[0] == 0
    assert rel_fro(on[1], off[1]) <= 2 * EPOCH_TOL and rel_fro(on[2], off[2]) <= 2 * EPOCH_TOL


def test_dense_mid_fit_rmse_matches_oracle(T):
    """Twenty epochs of the Zipf case with the automatic choice (which takes
    the tiles here), clip on: trajectory and held-out RMSE against the
    oracle's bf16 fit."""
    import paper_2608_00977_amd as tsid
    p = synth.mid()
    p.epochs, p.prec, p.clip = 20, "bf16", True
    note(f"dense mid fit nnz={p.nnz} k={p.k}")
    _build(T, p)
    st, P, Q, hist = gpu_fit(T, p, prec="bf16", clip=True)
    assert st == 0
    info = T.dense_info()
    _, _, a, b, v = oracle_template(p)
    assert info == _tile_info(a, b, p.I.size, p.J.size, auto_fill(p.k))  # the automatic rule took the tiles
    assert info["cells"] >= 0.10 * a.size
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, True, p.xi,
                                    bf16=True)
    assert sto == 0
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)
    want, n_test = oracle_rmse(Po, Qo, p)
    Tt = tsid.Tsid(0)
    try:
        Tt.build_template(p.m, p.n, p.tu, p.ti, p.tr, p.I, p.J, p.k)
        got = rmse_on(Tt, P, Q, n_test)
    finally:
        Tt.close()
    assert abs(got - want) <= BF16_RMSE_TOL * want, (got, want)


def test_dense_bitwise_repeatable_and_resumable(T):
    p, fill = _case("mid_zipf")
    _build(T, p)
    T.set_dense_tiles(fill)
    try:
        note("dense determinism")
        r1 = gpu_fit(T, p, epochs=10, prec="bf16")
        r2 = gpu_fit(T, p, epochs=10, prec="bf16")
        assert r1[0] == 0 and r2[0] == 0
        assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2])
        assert np.array_equal(r1[3], r2[3])
        h = gpu_fit(T, p, epochs=5, prec="bf16")
        h2 = gpu_fit(T, p, epochs=5, prec="bf16", P0=h[1], Q0=h[2])
        assert np.array_equal(h2[1], r1[1]) and np.array_equal(h2[2], r1[2])
    finally:
        T.set_dense_tiles(-1)


def test_dense_automatic_choice():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    try:
        p = synth.mid()
        _build(t, p)
        note("dense auto: mid fp32 / bf16")
        assert gpu_fit(t, p, epochs=1, prec="fp32")[0] == 0
        assert t.dense_info()["tiles"] == 0  # fp32 fits take no tiles
        assert gpu_fit(t, p, epochs=1, prec="bf16")[0] == 0
        assert t.dense_info()["cells"] > 0
        t.set_dense_tiles(0)
        assert gpu_fit(t, p, epochs=1, prec="bf16")[0] == 0
        assert t.dense_info()["tiles"] == 0
        t.set_dense_tiles(-1)
        # uniform cells at 1% density: no tile reaches 15%
        p = synth.random_case(3000, 2800, 90000, 1100, 900, 32, seed=36, epochs=1, prec="bf16")
        _build(t, p)
        note("dense auto: sparse uniform")
        assert gpu_fit(t, p, epochs=1, prec="bf16")[0] == 0
        assert t.dense_info()["tiles"] == 0
    finally:
        t.close()


def test_dense_rejects_unsupported(T):
    import paper_2608_00977_amd as tsid
    with pytest.raises(tsid.TsidError):
        T.set_dense_tiles(1.5)
    with pytest.raises(tsid.TsidError):
        T.set_dense_tiles(float("nan"))
    p, fill = _case("half_k32")
    _build(T, p)
    T.set_dense_tiles(fill)
    try:
        assert gpu_fit(T, p, epochs=1, prec="fp32")[0] == tsid.binding.E_INVAL
        p8 = synth.random_case(300, 280, 40000, 160, 140, 8, seed=37, epochs=1, prec="bf16")
        _build(T, p8)
        assert gpu_fit(T, p8, epochs=1, prec="bf16")[0] == tsid.binding.E_INVAL
    finally:
        T.set_dense_tiles(-1)
    # the automatic mode falls back to the item pass where tiles do not apply
    assert gpu_fit(T, p8, epochs=1, prec="bf16")[0] == 0
    assert T.dense_info()["tiles"] == 0


def test_dense_empty_template_is_pure_shrinkage(T):
    p, fill = _case("half_k32")
    p.u, p.i, p.r = p.u[:0], p.i[:0], p.r[:0]
    p.lam = 0.25
    _build(T, p)
    T.set_dense_tiles(fill)
    try:
        note("dense empty template")
        st, P, Q, _ = gpu_fit(T, p, epochs=4, prec="bf16", step="sum", lr=0.1)
        assert T.dense_info()["tiles"] == 0
    finally:
        T.set_dense_tiles(-1)
    assert st == 0
    np.testing.assert_allclose(P, p.P0.astype(np.float64) * 0.95 ** 4, rtol=1e-5)
    np.testing.assert_allclose(Q, p.Q0.astype(np.float64) * 0.95 ** 4, rtol=1e-5)


def test_dense_nonfinite_returns_last_finite_iterate(T):
    import paper_2608_00977_amd as tsid
    p, fill = _case("half_k32")
    _build(T, p)
    T.set_dense_tiles(fill)
    try:
        note("dense non-finite")
        st, P, Q, hist = gpu_fit(T, p, epochs=40, prec="bf16", step="sum", lr=30.0)
        assert st == tsid.binding.E_NONFINITE
        done = T.epochs_done()
        assert 0 < done < 40
        ref = gpu_fit(T, p, epochs=done, prec="bf16", step="sum", lr=30.0)
        assert ref[0] == 0
        assert np.array_equal(ref[1], P) and np.array_equal(ref[2], Q)
        assert np.all(np.isfinite(P)) and np.all(np.isfinite(Q))
        assert np.all(np.isnan(hist[done + 1:]))
    finally:
        T.set_dense_tiles(-1)


def test_dense_timing_reports_dense_kernels(T):
    p, fill = _case("mid_zipf")
    _build(T, p)
    T.set_dense_tiles(fill)
    T.set_timing(1)
    try:
        assert gpu_fit(T, p, epochs=3, prec="bf16")[0] == 0
        tm = T.timing()
    finally:
        T.set_timing(0)
        T.set_dense_tiles(-1)
    # both sides' tiles share one launch (and their combines another), as do the item passes
    assert tm["dense_launches"] == [3, 0]
    assert tm["pass_launches"] == [3, 0]
    assert tm["dense_ms"][0] > 0
    assert tm["epochs"] == 3
    assert tm["epoch_ms"] >= tm["dense_ms"][0] + tm["pass_ms"][0] + tm["pass_ms"][1] + tm["dense_ms"][1] - 1e-3
