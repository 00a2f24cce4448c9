"""Row-blocked Q passes (tsid_set_row_blocks) against the oracle, through the
C ABI.

The blocks change only which launch gathers which P rows and the order in
which a column's fp32 sums are added (per block, then the blocks in order),
so the full-gradient bars apply unchanged: fp32 factors within 1e-4
relative Frobenius error of the oracle, the loss trajectory within 1e-3;
bf16 with dense tiles one epoch within 1e-4 of the oracle's bf16 mode, as
the dense-tile tests do.  Cases: long (split) column buckets whose block
runs go through the fixup kernel, blocks without cells, more blocks than
needed, the similarity term's sums added by the combine kernel, and the
automatic choice (one block here).
"""
import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, oracle_template, rel_fro

pytestmark = pytest.mark.gpu

FP32_TOL = 1e-4
LOSS_TRAJ_TOL = 1e-3


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    t.set_pass_kernel("item")  # the slab pass has no row blocks
    yield t
    t.close()


def _case(name):
    if name == "ragged_k32":  # hot columns: long buckets, split over waves in every block
        return synth.random_case(700, 500, 9000, 300, 200, 32, seed=11, hot_rows=3, hot_cols=2, epochs=6,
                                 step="degree", lr=0.1)
    if name == "ragged_k8_sum":
        return synth.random_case(333, 257, 4000, 101, 77, 8, seed=12, hot_rows=1, epochs=5, step="sum",
                                 lr=0.02)
    if name == "ragged_k64":
        return synth.random_case(500, 450, 8000, 200, 180, 64, seed=14, hot_rows=2, hot_cols=1, epochs=4,
                                 step="degree", lr=0.1)
    if name == "ragged_k128_clip":
        return synth.random_case(300, 280, 6000, 160, 140, 128, seed=15, hot_rows=1, hot_cols=1, epochs=3,
                                 step="degree", lr=0.1, clip=True, xi=0.05)
    if name == "sparse_empty":  # most column buckets have no cell in most blocks
        return synth.random_case(2000, 1500, 600, 700, 500, 32, seed=16, epochs=4, step="degree", lr=0.05)
    raise KeyError(name)


def _fit(T, p, prec="fp32", epochs=None):
    import torch
    from paper_2608_00977_amd import make_opts
    P = torch.from_numpy(np.ascontiguousarray(p.P0, np.float32)).cuda()
    Q = torch.from_numpy(np.ascontiguousarray(p.Q0, np.float32)).cuda()
    opts = make_opts(epochs=p.epochs if epochs is None else epochs, lam=p.lam, lr=p.lr, clip=p.clip, xi=p.xi,
                     prec=prec, step=p.step)
    st, hist = T.fit_template(P, Q, opts, raise_on_error=False)
    return st, P.cpu().numpy(), Q.cpu().numpy(), hist


@pytest.mark.parametrize("name,nb", [("ragged_k32", 3), ("ragged_k32", 7), ("ragged_k8_sum", 4),
                                     ("ragged_k64", 2), ("ragged_k128_clip", 5), ("sparse_empty", 64)])
def test_row_blocked_fit_matches_oracle(T, name, nb):
    p = _case(name)
    note(f"row blocks {name} nb={nb} k={p.k}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_row_blocks(nb)
    try:
        st, P, Q, hist = _fit(T, p)
        used = T.row_blocks()
    finally:
        T.set_row_blocks(0)
    assert st == 0 and used == min(nb, p.I.size)
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, p.clip, p.xi)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL, rel_fro(P, Po)
    assert rel_fro(Q, Qo) <= FP32_TOL, rel_fro(Q, Qo)
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)


def test_row_blocks_bf16_dense_one_epoch(T):
    """bf16 with the automatic dense tiles: the blocked item Q pass walks the
    other cells, the combine adds the tile sums; one epoch against the
    oracle's bf16 mode (the dense-tile tests' bar)."""
    p = synth.mid()
    p.clip = True
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_row_blocks(4)
    try:
        note("row blocks bf16 mid")
        st, P, Q, _ = _fit(T, p, prec="bf16", epochs=1)
        assert st == 0 and T.row_blocks() == 4 and T.dense_info()["tiles"] > 0
    finally:
        T.set_row_blocks(0)
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, _, _ = oracle.fit(a, b, v, p.P0, p.Q0, 1, p.lam, p.lr, p.step, True, p.xi, bf16=True)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL and rel_fro(Q, Qo) <= FP32_TOL, (rel_fro(P, Po), rel_fro(Q, Qo))
    # another tile fill rebuilds the other cells' stream, and the blocks with it
    T.set_row_blocks(4)
    T.set_dense_tiles(0.5)
    try:
        note("row blocks bf16 mid, fill 0.5")
        st, P, Q, _ = _fit(T, p, prec="bf16", epochs=1)
        assert st == 0 and T.row_blocks() == 4 and T.dense_info()["tiles"] > 0
    finally:
        T.set_row_blocks(0)
        T.set_dense_tiles(-1)
    assert rel_fro(P, Po) <= FP32_TOL and rel_fro(Q, Qo) <= FP32_TOL, (rel_fro(P, Po), rel_fro(Q, Qo))


def test_row_blocks_with_similarity_term(T):
    p = _case("ragged_k32")
    A = np.random.default_rng(40).integers(0, 3, (p.J.size, 4))
    S = oracle.similarity(A)
    np.fill_diagonal(S, 0.0)
    r, c = np.nonzero(S >= 0.75)
    w = S[r, c].astype(np.float32)
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_similarity(r.astype(np.int32), c.astype(np.int32), w, 0.05)
    T.set_row_blocks(3)
    try:
        note("row blocks with the similarity term")
        st, P, Q, hist = _fit(T, p)
    finally:
        T.set_row_blocks(0)
        T.set_similarity(r.astype(np.int32), c.astype(np.int32), w, 0.0)
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit_mv(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, r, c, w, 0.05, p.step, p.clip,
                                       p.xi)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL and rel_fro(Q, Qo) <= FP32_TOL
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)


def test_row_blocks_repeatable_automatic_and_rejected(T):
    import paper_2608_00977_amd as tsid
    p = _case("ragged_k32")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    note("row blocks repeatable")
    T.set_row_blocks(3)
    try:
        r1 = _fit(T, p)
        r2 = _fit(T, p)
    finally:
        T.set_row_blocks(0)
    assert np.array_equal(r1[1], r2[1]) and np.array_equal(r1[2], r2[2]) and np.array_equal(r1[3], r2[3])
    # the P pass is untouched by the Q pass's blocks in the first epoch
    one_b = _fit(T, p, epochs=1)
    assert T.row_blocks() == 1  # a 24 KiB table: no blocks under the automatic rule
    T.set_row_blocks(3)
    try:
        one_a = _fit(T, p, epochs=1)
    finally:
        T.set_row_blocks(0)
    assert np.array_equal(one_a[1], one_b[1])
    assert rel_fro(one_a[2], one_b[2]) <= 1e-6
    for bad in (-1, 65):
        with pytest.raises(tsid.TsidError):
            T.set_row_blocks(bad)


def test_row_blocks_with_per_entry_clip_and_minibatch(T):
    """The per-entry clip's sums go through the block partials and the
    combine like the summed gradient's; mini-batch steps keep one pass."""
    import torch
    from paper_2608_00977_amd import make_opts
    p = _case("ragged_k32")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_row_blocks(3)
    try:
        note("row blocks with the per-entry clip")
        P = torch.from_numpy(np.ascontiguousarray(p.P0, np.float32)).cuda()
        Q = torch.from_numpy(np.ascontiguousarray(p.Q0, np.float32)).cuda()
        st, hist = T.fit_template(P, Q, make_opts(epochs=p.epochs, lam=p.lam, lr=p.lr, clip="per_entry", xi=0.05,
                                                  step=p.step), raise_on_error=False)
        assert st == 0 and T.row_blocks() == 3
        T.set_minibatch(2, 3)
        st2, *_ = _fit(T, p, epochs=1)
        assert st2 == 0 and T.row_blocks() == 1
    finally:
        T.set_minibatch(0)
        T.set_row_blocks(0)
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, p.step, 2, 0.05)
    assert sto == 0
    assert rel_fro(P.cpu().numpy(), Po) <= FP32_TOL and rel_fro(Q.cpu().numpy(), Qo) <= FP32_TOL
    np.testing.assert_allclose(hist, ho, rtol=LOSS_TRAJ_TOL)
