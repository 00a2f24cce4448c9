"""Mini-batch epochs (tsid_set_minibatch; the in-epoch updates of Section 5.1
grouped into batches) against the oracle's fit_minibatch on the same seeded
inputs, through the C ABI.

Bars: the batch pointers bit-exact (the batch of every cell is an integer
decision, taken on both sides from the same 64-bit hash); fp32 factors within
1e-4 relative Frobenius error of the fp64 oracle after a fixed number of
epochs, the loss trajectory within 1e-3 and the final loss within 1e-6 of the
oracle's Eq. 2 at the library's own factors, as for the full-gradient fit
(each batch step is one such fit's step on fewer cells); bf16 factors
within 1e-2 relative held-out RMSE.
"""
import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, oracle_rmse, oracle_template, rel_fro, rmse_on

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
    if name == "ragged_k32_B4":  # hot lines longer than an item: split buckets in every batch
        return synth.random_case(700, 500, 9000, 300, 200, 32, seed=11, hot_rows=3, hot_cols=2,
                                 epochs=6, step="degree", lr=0.1), 4, 7
    if name == "ragged_k8_sum_B3":
        return synth.random_case(333, 257, 4000, 101, 77, 8, seed=12, hot_rows=1, epochs=5,
                                 step="sum", lr=0.02), 3, 1
    if name == "ragged_k16_B7":
        return synth.random_case(400, 300, 5000, 150, 120, 16, seed=13, hot_cols=2, epochs=4,
                                 step="degree", lr=0.1), 7, 2
    if name == "ragged_k64_B2":
        return synth.random_case(500, 450, 8000, 200, 180, 64, seed=14, hot_rows=2, hot_cols=1,
                                 epochs=4, step="degree", lr=0.1), 2, 3
    if name == "ragged_k128_clip_B5":
        return synth.random_case(300, 280, 6000, 160, 140, 128, seed=15, hot_rows=1, hot_cols=1,
                                 epochs=3, step="degree", lr=0.1, clip=True, xi=0.05), 5, 4
    if name == "sparse_empty_B6":  # most lines have no cell in a given batch
        return synth.random_case(2000, 1500, 600, 700, 500, 32, seed=16, epochs=4,
                                 step="degree", lr=0.05), 6, 5
    if name == "tiny_B2":
        return synth.tiny(), 2, 6
    raise KeyError(name)


CASES = ["ragged_k32_B4", "ragged_k8_sum_B3", "ragged_k16_B7", "ragged_k64_B2", "ragged_k128_clip_B5",
         "sparse_empty_B6", "tiny_B2"]


def _build(T, p):
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)


def _fit(T, p, prec="fp32", epochs=None, lr=None, P0=None, Q0=None):
    import torch
    from paper_2608_00977_amd import make_opts
    P = torch.from_numpy(np.ascontiguousarray(p.P0 if P0 is None else P0, np.float32)).cuda()
    Q = torch.from_numpy(np.ascontiguousarray(p.Q0 if Q0 is None else Q0, np.float32)).cuda()
    opts = make_opts(epochs=p.epochs if epochs is None else epochs, lam=p.lam, lr=p.lr if lr is None else lr,
                     clip=p.clip, xi=p.xi, prec=prec, step=p.step)
    st, hist = T.fit_template(P, Q, opts, raise_on_error=False)
    return st, P.cpu().numpy(), Q.cpu().numpy(), hist


def _expected_batch_ptr(a, b, rows, side, B, seed):
    """Batch pointers from the oracle's batch rule: counts per (batch, owner
    line), prefix-summed."""
    own = b if side else a
    beta = np.array([oracle.batch_of(x, y, seed, B) for x, y in zip(a, b)], np.int64)
    cnt = np.bincount(beta * rows + own, minlength=B * rows)
    return np.concatenate([[0], np.cumsum(cnt)]).astype(np.int64)


@pytest.mark.parametrize("name", ["ragged_k32_B4", "sparse_empty_B6"])
def test_batch_pointers_bit_exact(T, name):
    p, B, seed = _case(name)
    note(f"minibatch pointers {name} B={B}")
    _build(T, p)
    T.set_minibatch(B, seed)
    try:
        st, *_ = _fit(T, p, epochs=0)
        assert st == 0
        _, _, a, b, v = oracle_template(p)
        assert np.array_equal(T.export_index("batch_ptr_r"), _expected_batch_ptr(a, b, p.I.size, 0, B, seed))
        assert np.array_equal(T.export_index("batch_ptr_c"), _expected_batch_ptr(a, b, p.J.size, 1, B, seed))
    finally:
        T.set_minibatch(0)


@pytest.mark.parametrize("name", CASES)
def test_minibatch_fit_fp32_matches_oracle(T, name):
    p, B, seed = _case(name)
    note(f"minibatch fp32 {name} B={B} k={p.k} epochs={p.epochs} step={p.step}")
    _build(T, p)
    T.set_minibatch(B, seed)
    try:
        st, P, Q, hist = _fit(T, p)
    finally:
        T.set_minibatch(0)
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, done = oracle.fit_minibatch(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, p.clip,
                                                 p.xi, n_batches=B, seed=seed)
    assert sto == 0 and done == p.epochs
    assert rel_fro(P, Po) <= FP32_TOL, rel_fro(P, Po)
    assert rel_fro(Q, Qo) <= FP32_TOL, rel_fro(Q, Qo)
    at_gpu = oracle.loss(a, b, v, p.I.size, p.J.size, P, Q, p.lam)
    assert abs(hist[-1] - at_gpu) <= LOSS_KERNEL_TOL * at_gpu
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)


@pytest.mark.parametrize("prec", ["fp32", "bf16"])
def test_one_batch_is_the_full_gradient_fit(T, prec):
    """With one batch the steps are the Jacobi fit's (item pass, same plan):
    the factors of every line with a cell match bit for bit; lines without a
    cell keep their start rows instead of shrinking."""
    p, _, _ = _case("sparse_empty_B6")
    _build(T, p)
    T.set_pass_kernel("item")
    T.set_dense_tiles(0)
    try:
        note(f"minibatch one batch {prec}")
        st, Pj, Qj, hj = _fit(T, p, prec=prec)
        T.set_minibatch(1, 99)
        st2, P1, Q1, h1 = _fit(T, p, prec=prec)
    finally:
        T.set_minibatch(0)
        T.set_pass_kernel("auto")
        T.set_dense_tiles(-1)
    assert st == st2 == 0
    dr, dc = T.export_index("deg_r") > 0, T.export_index("deg_c") > 0
    assert (~dr).any() or (~dc).any(), "the case should have lines without cells"
    assert np.array_equal(P1[dr], Pj[dr]) and np.array_equal(Q1[dc], Qj[dc])
    assert np.array_equal(P1[~dr], p.P0[~dr].astype(np.float32))
    assert np.array_equal(Q1[~dc], p.Q0[~dc].astype(np.float32))
    assert h1[0] == pytest.approx(hj[0], rel=1e-6)


def test_minibatch_bf16_rmse_matches_oracle(T):
    """bf16 factors with fp32 accumulation and the clip: held-out RMSE within
    1e-2 relative of the oracle's (fp64 master, bf16-rounded products)."""
    p = synth.mid()
    p.clip, p.lr = True, 0.05
    B, seed = 4, 8
    note(f"minibatch bf16 mid B={B} nnz={p.nnz} k={p.k} epochs={p.epochs}")
    _build(T, p)
    T.set_minibatch(B, seed)
    try:
        st, P, Q, _ = _fit(T, p, prec="bf16")
    finally:
        T.set_minibatch(0)
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, _, _ = oracle.fit_minibatch(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, True, p.xi,
                                             bf16=True, n_batches=B, seed=seed)
    assert sto == 0
    r_gpu, _ = oracle_rmse(P.astype(np.float64), Q.astype(np.float64), p)
    r_or, _ = oracle_rmse(Po, Qo, p)
    assert abs(r_gpu - r_or) <= BF16_RMSE_TOL * r_or, (r_gpu, r_or)


def test_minibatch_repeatable_and_seed_dependent(T):
    """Fixed orders, no atomics: the same seed gives the same bits; another
    seed deals other batches and ends elsewhere; batch count 0 restores the
    full-gradient fit."""
    p, B, seed = _case("ragged_k32_B4")
    _build(T, p)
    note("minibatch repeatable")
    st, Pj, Qj, _ = _fit(T, p)
    T.set_minibatch(B, seed)
    try:
        r1 = _fit(T, p)
        r2 = _fit(T, p)
        T.set_minibatch(B, seed + 1)
        r3 = _fit(T, p)
    finally:
        T.set_minibatch(0)
    r4 = _fit(T, p)
    assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2])
    assert np.array_equal(r1[3], r2[3], equal_nan=True)
    assert not np.array_equal(r1[1], r3[1])
    assert np.array_equal(r4[1], Pj) and np.array_equal(r4[2], Qj)


def test_minibatch_nonfinite_stops_with_whole_epochs(T):
    import paper_2608_00977_amd as tsid
    p = synth.random_case(200, 150, 2000, 64, 48, 32, seed=5, step="sum")
    _build(T, p)
    T.set_minibatch(3, 2)
    try:
        note("minibatch non-finite")
        st, P, Q, hist = _fit(T, p, epochs=60, lr=50.0)
        assert st == tsid.binding.E_NONFINITE
        done = T.epochs_done()
        assert 0 <= done < 60 and np.all(np.isfinite(P)) and np.all(np.isfinite(Q))
        # (the fp32 loss of the huge iterates may itself overflow: only the
        # entries after the last whole epoch are defined to be NaN)
        assert np.isfinite(hist[0]) and np.all(np.isnan(hist[done + 1:]))
        st2, _, _, h2 = _fit(T, p, epochs=done, lr=50.0)
        assert st2 == 0 and T.epochs_done() == done
        np.testing.assert_array_equal(h2, hist[:done + 1])
    finally:
        T.set_minibatch(0)
    # the fp64 oracle leaves the finite range too, no earlier than fp32
    _, _, a, b, v = oracle_template(p)
    sto, _, _, _, done_o = oracle.fit_minibatch(a, b, v, p.P0, p.Q0, 60, p.lam, 50.0, "sum", n_batches=3, seed=2)
    assert sto == 7 and done_o >= done


def test_minibatch_rejections_and_timing(T):
    import paper_2608_00977_amd as tsid
    p, B, seed = _case("ragged_k16_B7")
    _build(T, p)
    with pytest.raises(tsid.TsidError):
        T.set_minibatch(-1)
    with pytest.raises(tsid.TsidError):
        T.set_minibatch(4097)
    T.set_minibatch(B, seed)
    try:
        T.set_pass_kernel("slab")
        st, *_ = _fit(T, p, epochs=1)
        assert st == tsid.binding.E_INVAL
        T.set_pass_kernel("auto")
        T.set_dense_tiles(0.2)
        st, *_ = _fit(T, p, prec="bf16", epochs=1)
        assert st == tsid.binding.E_INVAL
        T.set_dense_tiles(-1)
        note("minibatch timing")
        T.set_timing(1)
        st, *_ = _fit(T, p, epochs=3)
        tm = T.timing()
        assert st == 0 and tm["epochs"] == 3 and tm["epoch_ms"] > 0
        assert tm["pass_launches"] == [3, 3] and tm["dense_launches"] == [0, 0]
    finally:
        T.set_timing(0)
        T.set_pass_kernel("auto")
        T.set_dense_tiles(-1)
        T.set_minibatch(0)
