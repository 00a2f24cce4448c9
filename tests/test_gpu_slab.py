"""Parity of the slab pass kernel (one lane per factor row, the other factor
staged through LDS in slabs of 128 KiB) with the fp64 oracle, through the C
ABI.

The slab pass computes the same epochs as the item pass (Eqs. 2-5, Section
5.3); these tests force it on every fp32 rank it supports, on cases with
several row blocks, several slabs with a ragged last slab, blocks split over
several workgroups (partial sums added by the finishing kernel), long
buckets, and many short or empty runs (the pass's record copy pads every
run to whole blocks of eight, and odd rows walk their runs backwards).
Bars as for the item pass: factors within 1e-4 relative Frobenius error, the
loss of the final iterate within 1e-6, the trajectory within 1e-3, results
bitwise repeatable.
"""
import os

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import gpu_fit, note, oracle_template, rel_fro

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
LOSS_KERNEL_TOL = 1e-6
LOSS_TRAJ_TOL = 1e-3


def _case(name):
    if name == "tiny":  # k = 8: one block, one slab
        return synth.tiny()
    if name == "blocks_k32":  # P pass: 3 blocks of 512 rows (the last 76), 3 slabs of 1024
        return synth.random_case(3000, 2800, 300000, 1100, 2600, 32, seed=21, epochs=8,
                                 step="degree", lr=0.2)  # rows (the last 552); Q pass: 6 x 2
    if name == "hot_k32":  # whole rows and columns observed: buckets far longer than the rest
        return synth.random_case(700, 500, 9000, 300, 200, 32, seed=11, hot_rows=3, hot_cols=2,
                                 epochs=12, step="degree", lr=0.1)
    if name == "k16_sum":
        return synth.random_case(1500, 1400, 60000, 600, 1300, 16, seed=22, epochs=6,
                                 step="sum", lr=0.01)
    if name == "k64_clip":  # 4 slabs of 512 rows per pass
        return synth.random_case(2200, 2100, 250000, 2000, 1900, 64, seed=23, epochs=5,
                                 step="degree", lr=0.1, clip=True, xi=0.05)
    if name == "k8_sparse":  # many empty buckets
        return synth.random_case(2000, 1500, 600, 700, 500, 8, seed=16, epochs=5,
                                 step="degree", lr=0.05)
    raise KeyError(name)


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    t.set_pass_kernel("slab")
    yield t
    t.close()


def _build(T, p):
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)


def _check_fit(T, p):
    st, P, Q, hist = gpu_fit(T, p, prec="fp32")
    assert st == 0
    assert T.pass_kernels() == ("slab", "slab")
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, p.clip, p.xi)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL, rel_fro(P, Po)
    assert rel_fro(Q, Qo) <= FP32_TOL, rel_fro(Q, Qo)
    at_gpu = oracle.loss(a, b, v, p.I.size, p.J.size, P, Q, p.lam)
    assert abs(hist[-1] - at_gpu) <= LOSS_KERNEL_TOL * at_gpu
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)
    return P, Q


@pytest.mark.parametrize("name", ["tiny", "blocks_k32", "hot_k32", "k16_sum", "k64_clip", "k8_sparse"])
def test_slab_fit_matches_oracle(T, name):
    p = _case(name)
    note(f"slab fit {name} k={p.k} nnz={p.nnz} m_t={p.I.size} n_t={p.J.size}")
    _build(T, p)
    _check_fit(T, p)


@pytest.mark.parametrize("units", ["1", "6", "4096"])
def test_slab_unit_split_does_not_change_parity(units):
    """The split of a block's slabs over workgroups (P pass: one workgroup per
    block; two workgroups of two slabs and one; three of one slab) changes
    only the order of the partial sums."""
    import paper_2608_00977_amd as tsid
    old = os.environ.get("TSID_SLAB_UNITS")
    os.environ["TSID_SLAB_UNITS"] = units
    t = tsid.Tsid(0)
    try:
        t.set_pass_kernel("slab")
        p = _case("blocks_k32")
        note(f"slab units={units}")
        _build(t, p)
        _check_fit(t, p)
    finally:
        t.close()
        if old is None:
            os.environ.pop("TSID_SLAB_UNITS", None)
        else:
            os.environ["TSID_SLAB_UNITS"] = old


def test_slab_bitwise_repeatable_and_resumable(T):
    p = _case("blocks_k32")
    _build(T, p)
    note("slab determinism")
    r1 = gpu_fit(T, p, epochs=10)
    r2 = gpu_fit(T, p, epochs=10)
    assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2])
    assert np.array_equal(r1[3], r2[3])
    h = gpu_fit(T, p, epochs=5)
    h2 = gpu_fit(T, p, epochs=5, P0=h[1], Q0=h[2])
    assert np.array_equal(h2[1], r1[1]) and np.array_equal(h2[2], r1[2])


def test_auto_picks_slab_for_even_templates_and_item_otherwise():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    try:
        p = _case("blocks_k32")  # uniform cells, fp32
        _build(t, p)
        note("auto: uniform fp32")
        assert gpu_fit(t, p, epochs=1)[0] == 0
        assert t.pass_kernels() == ("slab", "slab")
        note("auto: uniform bf16")
        assert gpu_fit(t, p, epochs=1, prec="bf16")[0] == 0
        assert t.pass_kernels() == ("item", "item")
        p = _case("hot_k32")  # a few whole rows / columns: buckets far above the mean
        _build(t, p)
        note("auto: hot buckets")
        assert gpu_fit(t, p, epochs=1)[0] == 0
        assert t.pass_kernels() == ("item", "item")
    finally:
        t.close()


def test_slab_and_item_agree(T):
    """Both kernels on the same template: each within the oracle bar, so
    within 2e-4 of each other."""
    import paper_2608_00977_amd as tsid
    p = _case("k64_clip")
    _build(T, p)
    note("slab vs item")
    a = gpu_fit(T, p)
    t = tsid.Tsid(0)
    try:
        t.set_pass_kernel("item")
        _build(t, p)
        b = gpu_fit(t, p)
        assert t.pass_kernels() == ("item", "item")
    finally:
        t.close()
    assert rel_fro(a[1], b[1]) <= 2 * FP32_TOL and rel_fro(a[2], b[2]) <= 2 * FP32_TOL


def test_slab_rejects_unsupported_rank_and_precision(T):
    import paper_2608_00977_amd as tsid
    p = _case("hot_k32")
    _build(T, p)
    st, _, _, _ = gpu_fit(T, p, epochs=1, prec="bf16")
    assert st == tsid.binding.E_INVAL
    p = synth.random_case(300, 280, 6000, 160, 140, 128, seed=15, epochs=1)
    _build(T, p)
    st, _, _, _ = gpu_fit(T, p, epochs=1)
    assert st == tsid.binding.E_INVAL


def test_slab_nonfinite_returns_last_finite_iterate(T):
    """A step size that overflows: the fit stops at the first non-finite
    epoch and returns the iterate before it, as the item pass does."""
    import paper_2608_00977_amd as tsid
    p = _case("blocks_k32")
    _build(T, p)
    note("slab non-finite")
    st, P, Q, hist = gpu_fit(T, p, epochs=40, step="sum", lr=30.0)
    assert st == tsid.binding.E_NONFINITE
    done = T.epochs_done()
    assert 0 < done < 40
    ref = gpu_fit(T, p, epochs=done, step="sum", lr=30.0)
    assert ref[0] == 0
    assert np.array_equal(ref[1], P) and np.array_equal(ref[2], Q)
    assert np.all(np.isfinite(P)) and np.all(np.isfinite(Q))
    assert np.all(np.isnan(hist[done + 1:]))


def test_slab_passes_share_one_launch(T):
    """With the slab pass on both sides the P and Q passes of an epoch go out
    as one launch, and their finishing kernels as another (the Q pass reads
    only the old factors); the kernel timer sees one pass launch per timed
    epoch, counted as the P pass, and one finish."""
    p = _case("blocks_k32")
    _build(T, p)
    note("slab pair launch")
    T.set_timing(2)
    try:
        st, P, Q, hist = gpu_fit(T, p, prec="fp32", epochs=6)
        tm = T.timing()
    finally:
        T.set_timing(0)
    assert st == 0 and T.pass_kernels() == ("slab", "slab")
    assert tm["pass_launches"] == [3, 0] and tm["fixup_launches"] == 3 and tm["epochs"] == 3
    assert tm["epoch_ms"] >= tm["pass_ms"][0] + tm["fixup_ms"] - 1e-3
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, 6, p.lam, p.lr, p.step, p.clip, p.xi)
    assert sto == 0 and rel_fro(P, Po) <= FP32_TOL and rel_fro(Q, Qo) <= FP32_TOL
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)
