"""The step scale and clip order options (tsid_step COL_DEGREE, clip 3)
through the C ABI.

Two kinds of check:
- the hand-derived epochs of tests/golden/hand_steps.json run through the
  library itself (k = 8, the fixture's single coordinate followed by seven
  zero coordinates, which stay zero), compared with the fixture's values,
  which no code produced: these pin the library to the printed forms of
  Eq. 5 and Section 5.3 without going through the oracle;
- ragged parity cases of every pass kernel (item pass with split buckets
  and the fixup, slab pass, row-blocked Q pass, bf16 dense tiles) against
  the oracle with the same options, at the bars of the other parity tests
  (fp32 factors 1e-4 relative Frobenius error after the epochs; one bf16
  epoch with dense tiles 1e-4).
"""
import json
import os

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import gpu_fit, note, oracle_template, rel_fro

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_steps.json")
FP32_TOL = 1e-4
K_PAD = 8


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    yield t
    t.set_pass_kernel("auto")
    t.close()


def _pad(x):
    x = np.asarray(x, np.float32).reshape(-1, 1)
    return np.concatenate([x, np.zeros((x.shape[0], K_PAD - 1), np.float32)], axis=1)


def _run(T, m, n, u, i, r, P0, Q0, epochs, lam, lr, step, clip, xi, prec="fp32"):
    import torch
    from paper_2608_00977_amd import make_opts
    T.build_template(m, n, np.asarray(u, np.int32), np.asarray(i, np.int32), np.asarray(r, np.float32),
                     np.arange(m, dtype=np.int32), np.arange(n, dtype=np.int32), K_PAD)
    P = torch.from_numpy(_pad(P0)).cuda()
    Q = torch.from_numpy(_pad(Q0)).cuda()
    opts = make_opts(epochs=epochs, lam=lam, lr=lr, clip={0: False, 1: True, 3: "printed"}[clip], xi=xi,
                     prec=prec, step=step)
    st, hist = T.fit_template(P, Q, opts)
    return st, P.cpu().numpy(), Q.cpu().numpy(), hist


@pytest.mark.parametrize("kernel", ["item", "slab"])
def test_golden_step_scale_and_clip_order(T, kernel):
    g = json.load(open(GOLDEN))["two_lines"]
    cells = np.array(g["cells"])
    T.set_pass_kernel(kernel)
    for c in g["cases"]:
        note(f"golden two_lines {c['name']} kernel={kernel}")
        st, P, Q, hist = _run(T, 2, 2, cells[:, 0], cells[:, 1], cells[:, 2], np.ravel(g["P"]),
                              np.ravel(g["Q"]), 1, c["lambda"], g["lr"], c["step"], c["clip"], c["xi"])
        assert st == 0
        assert T.pass_kernels() == (kernel, kernel)
        np.testing.assert_allclose(P[:, 0], np.ravel(c["P1"]), rtol=1e-6, err_msg=c["name"])
        np.testing.assert_allclose(Q[:, 0], np.ravel(c["Q1"]), rtol=1e-6, err_msg=c["name"])
        assert not P[:, 1:].any() and not Q[:, 1:].any()
        assert hist[0] == pytest.approx(c["loss0"], rel=1e-6)
    T.set_pass_kernel("auto")


def test_golden_bf16_epoch(T):
    """The library's bf16 mode on the hand-derived epoch: products from RNE
    bf16 copies, the fp32 master updated and used in the regulariser."""
    c = json.load(open(GOLDEN))["bf16"]
    note("golden bf16 epoch")
    T.set_pass_kernel("item")
    st, P, Q, hist = _run(T, 1, 1, [0], [0], [c["r"]], [c["p"]], [c["q"]], 1, c["lambda"], c["lr"], c["step"],
                          c["clip"], c["xi"], prec="bf16")
    T.set_pass_kernel("auto")
    assert st == 0
    assert P[0, 0] == pytest.approx(c["p1"], rel=1e-6)
    assert Q[0, 0] == pytest.approx(c["q1"], rel=1e-6)
    assert hist[0] == pytest.approx(c["loss0"], rel=1e-6)


OPTIONS = [("degree", "printed"), ("col_degree", False), ("col_degree", "printed"), ("col_degree", True)]


def _ragged(k, seed, prec="fp32"):
    # hot rows and columns longer than a work item (split buckets, fixups)
    return synth.random_case(700, 500, 9000, 300, 200, k, seed=seed, hot_rows=3, hot_cols=2, epochs=8,
                             step="degree", lr=0.02, prec=prec, xi=0.05)


@pytest.mark.parametrize("kernel", ["item", "slab"])
@pytest.mark.parametrize("step,clip", OPTIONS)
def test_options_match_oracle(T, kernel, step, clip):
    p = _ragged(32, 61)
    note(f"update options step={step} clip={clip} kernel={kernel} nnz={p.nnz}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_pass_kernel(kernel)
    try:
        st, P, Q, hist = gpu_fit(T, p, step=step, clip=clip)
        assert T.pass_kernels() == (kernel, kernel)
    finally:
        T.set_pass_kernel("auto")
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    sto, Po, Qo, ho, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, step, clip, p.xi)
    assert sto == 0
    assert rel_fro(P, Po) <= FP32_TOL and rel_fro(Q, Qo) <= FP32_TOL, (rel_fro(P, Po), rel_fro(Q, Qo))
    if clip:  # the clip is active: the two orders end apart
        other = {True: "printed", "printed": True}[clip]
        _, Px, Qx, _, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, step, other, p.xi)
        assert rel_fro(Px, Po) > 1e-3 or rel_fro(Qx, Qo) > 1e-3


@pytest.mark.parametrize("step,clip", [("degree", "printed"), ("col_degree", "printed")])
def test_options_row_blocks_match_oracle(T, step, clip):
    """The row-blocked Q pass applies the update in its combine kernel."""
    p = _ragged(64, 62)
    note(f"update options row blocks step={step} clip={clip}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_pass_kernel("item")
    T.set_row_blocks(4)
    try:
        st, P, Q, _ = gpu_fit(T, p, step=step, clip=clip)
        assert T.row_blocks() == 4
    finally:
        T.set_row_blocks(0)
        T.set_pass_kernel("auto")
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    _, Po, Qo, _, _ = oracle.fit(a, b, v, p.P0, p.Q0, p.epochs, p.lam, p.lr, step, clip, p.xi)
    assert rel_fro(P, Po) <= FP32_TOL and rel_fro(Q, Qo) <= FP32_TOL, (rel_fro(P, Po), rel_fro(Q, Qo))


@pytest.mark.parametrize("step,clip", [("degree", "printed"), ("col_degree", "printed")])
def test_options_bf16_dense_tiles_one_epoch(T, step, clip):
    """bf16 with the dense head tiles: one epoch against the oracle's bf16
    mode (both round the same fp32 start to bf16), as the dense-tile tests."""
    p = synth.random_case(350, 330, 57000, 211, 177, 64, seed=63, hot_cols=2, epochs=1, step="degree", lr=0.2,
                          prec="bf16", clip=True, xi=0.05)
    note(f"update options bf16 dense step={step} clip={clip}")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    T.set_dense_tiles(0.5)
    try:
        st, P, Q, _ = gpu_fit(T, p, epochs=1, prec="bf16", step=step, clip=clip)
        assert T.dense_info()["tiles"] > 0
    finally:
        T.set_dense_tiles(-1)
    assert st == 0
    _, _, a, b, v = oracle_template(p)
    _, Po, Qo, _, _ = oracle.fit(a, b, v, p.P0, p.Q0, 1, p.lam, p.lr, step, clip, p.xi, bf16=True)
    assert rel_fro(P, Po) <= 1e-4 and rel_fro(Q, Qo) <= 1e-4, (rel_fro(P, Po), rel_fro(Q, Qo))


def test_extension_clip_printed_and_column_step(T):
    """The extension takes clip 3 and rejects the column-only step (a
    template-fit option, E_INVAL)."""
    import torch
    from paper_2608_00977_amd import TsidError, make_opts
    g = synth.make_rng(64, "cells")
    k, n_fixed, n_free, nnz = 32, 400, 300, 6000
    F = g.standard_normal((n_fixed, k)).astype(np.float32) * 0.3
    fixed = g.integers(0, n_fixed, nnz).astype(np.int32)
    free = g.integers(0, n_free, nnz).astype(np.int32)
    key = np.unique(free.astype(np.int64) * n_fixed + fixed)
    free, fixed = (key // n_fixed).astype(np.int32), (key % n_fixed).astype(np.int32)
    r = g.standard_normal(key.size).astype(np.float32)
    p = synth.tiny()
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, k)
    note("extension clip printed")
    Fd = torch.from_numpy(F).cuda()
    out = torch.zeros((n_free, k), dtype=torch.float32).pin_memory()
    opts = make_opts(epochs=10, lam=0.01, lr=0.05, clip="printed", xi=0.05, step="degree")
    T.extend_chunk(1, fixed, free, r, n_free, Fd, out, opts)
    T.sync()
    st, Xo = oracle.extend(fixed, free, r, n_free, F, 10, 0.01, 0.05, "degree", "printed", 0.05)
    assert st == 0
    assert rel_fro(out.numpy(), Xo) <= FP32_TOL
    with pytest.raises(TsidError) as e:
        T.extend_chunk(1, fixed, free, r, n_free, Fd, out,
                       make_opts(epochs=3, lam=0.01, lr=0.05, step="col_degree"))
    assert e.value.status == 1  # TSID_E_INVAL
