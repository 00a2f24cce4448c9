"""The per-entry order of the clipped update (fit option clip = 2; Section 5.3
applied to Eqs. 3-4 entry by entry, before the 1/n average of Eq. 5) against
the oracle's clip mode 2, through the C ABI.

Each cell adds min(2 e q - 2 lambda p, xi) per coordinate; min is
piecewise linear with slope at most 1, so the fp32 library and the fp64
oracle stay as close as in the unclipped fit.  Bars: the full-gradient fit's
(fp32 factors within 1e-4 relative Frobenius error, loss trajectory within
1e-3, final loss within 1e-6 at the library's own factors; bf16 held-out RMSE
within 1e-2), for Jacobi and mini-batch epochs.
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


def _case(name):
    if name == "ragged_k32":  # split buckets (fixup) and active clips
        return synth.random_case(700, 500, 9000, 300, 200, 32, seed=11, hot_rows=3, hot_cols=2, epochs=6,
                                 step="degree", lr=0.1, clip=True, xi=0.05)
    if name == "ragged_k8_sum":
        # (each cell may add up to xi: the sum step of a long line needs a small lr)
        return synth.random_case(333, 257, 4000, 101, 77, 8, seed=12, hot_rows=1, epochs=5, step="sum",
                                 lr=0.005, clip=True, xi=0.1)
    if name == "ragged_k64":
        return synth.random_case(500, 450, 8000, 200, 180, 64, seed=14, hot_rows=2, hot_cols=1, epochs=4,
                                 step="degree", lr=0.1, clip=True, xi=0.02)
    if name == "ragged_k128":
        return synth.random_case(300, 280, 6000, 160, 140, 128, seed=15, hot_rows=1, hot_cols=1, epochs=3,
                                 step="degree", lr=0.1, clip=True, xi=0.05)
    if name == "sparse_empty":  # lines without cells stay where they are
        return synth.random_case(2000, 1500, 600, 700, 500, 32, seed=16, epochs=4, step="degree", lr=0.05,
                                 clip=True, xi=0.05)
    raise KeyError(name)


def _fit(T, p, prec="fp32", epochs=None):
    import torch
    from paper_2608_00977_amd import make_opts
    P = torch.from_numpy(np.ascontiguousarray(p.P0, np.float32)).cuda()
    Q = torch.from_numpy(np.ascontiguousarray(p.Q0, np.float32)).cuda()
    opts = make_opts(epochs=p.epochs if epochs is None else epochs, lam=p.lam, lr=p.lr, clip="per_entry",
                     xi=p.xi, prec=prec, step=p.step)
    st, hist = T.fit_template(P, Q, opts, raise_on_error=False)
    return st, P.cpu().numpy(), Q.cpu().numpy(), hist


def _check(p, P, Q, hist, sto, Po, Qo, ho):
    _, _, a, b, v = oracle_template(p)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL, rel_fro(P, Po)
    assert rel_fro(Q, Qo) <= FP32_TOL, rel_fro(Q, Qo)
    at_gpu = oracle.loss(a, b, v, p.I.size, p.J.size, P, Q, p.lam)
    assert abs(hist[-1] - at_gpu) <= LOSS_KERNEL_TOL * at_gpu
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)


@pytest.mark.parametrize("name", ["ragged_k32", "ragged_k8_sum", "ragged_k64", "ragged_k128", "sparse_empty"])
def test_per_entry_clip_fit_matches_oracle(T, name):
    p = _case(name)
    note(f"per-entry clip {name} k={p.k} xi={p.xi} step={p.step}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    st, P, Q, hist = _fit(T, p)
    assert st == 0 and T.pass_kernels() == ("item", "item")
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, 2, p.xi)
    _check(p, P, Q, hist, sto, Po, Qo, ho)
    if name == "sparse_empty":
        dr = np.bincount(a, minlength=p.I.size) == 0
        assert dr.any() and np.array_equal(P[dr], p.P0[dr].astype(np.float32))
    # the clip is active: the per-entry order moves elsewhere than the summed clip
    st1, P1, *_ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, 1, p.xi)
    assert rel_fro(Po, P1) > 10 * FP32_TOL


@pytest.mark.parametrize("name,B,seed", [("ragged_k32", 4, 3), ("ragged_k8_sum", 3, 5)])
def test_per_entry_clip_minibatch_matches_oracle(T, name, B, seed):
    p = _case(name)
    note(f"per-entry clip minibatch {name} B={B}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_minibatch(B, seed)
    try:
        st, P, Q, hist = _fit(T, p)
    finally:
        T.set_minibatch(0)
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit_minibatch(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, 2, p.xi,
                                              n_batches=B, seed=seed)
    _check(p, P, Q, hist, sto, Po, Qo, ho)


def test_per_entry_clip_bf16_rmse_matches_oracle(T):
    p = synth.mid()
    p.lr, p.xi = 0.05, 0.05
    note(f"per-entry clip bf16 mid nnz={p.nnz} k={p.k}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    st, P, Q, _ = _fit(T, p, prec="bf16")
    assert st == 0 and T.dense_info()["tiles"] == 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, _, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, 2, p.xi, bf16=True)
    assert sto == 0
    r_gpu, _ = oracle_rmse(P.astype(np.float64), Q.astype(np.float64), p)
    r_or, _ = oracle_rmse(Po, Qo, p)
    assert abs(r_gpu - r_or) <= BF16_RMSE_TOL * r_or, (r_gpu, r_or)


def test_per_entry_clip_rejections(T):
    import torch
    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd import make_opts
    p = _case("ragged_k32")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    note("per-entry clip rejections")
    try:
        T.set_pass_kernel("slab")
        assert _fit(T, p, epochs=1)[0] == tsid.binding.E_INVAL
        T.set_pass_kernel("auto")
        T.set_dense_tiles(0.2)
        assert _fit(T, p, prec="bf16", epochs=1)[0] == tsid.binding.E_INVAL
    finally:
        T.set_pass_kernel("auto")
        T.set_dense_tiles(-1)
    F = torch.zeros((10, p.k), dtype=torch.float32).cuda()
    out = torch.empty((1, p.k), dtype=torch.float32).pin_memory()
    with pytest.raises(tsid.TsidError) as ei:
        T.extend_chunk(0, np.zeros(1, np.int32), np.zeros(1, np.int32), np.ones(1, np.float32), 1, F, out,
                       make_opts(epochs=2, lam=0.1, lr=0.1, clip="per_entry", xi=0.1))
    assert ei.value.status == tsid.binding.E_INVAL
