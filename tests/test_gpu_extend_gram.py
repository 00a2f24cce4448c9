"""One-sided extension steps in Gram form (tsid_extend_chunk; Section 5.2 with
Eq. 5's update), through the C ABI.

A free row whose cells number at least the Gram threshold is stepped from its
fp64 Gram matrix and right-hand side (the gradient 2 lambda x - 2 (b - G x)),
the others by the per-cell kernel in fp32.  The oracle (or_extend, fp64)
takes every step cell by cell, so the Gram rows differ from it only in the
order of fp64 sums and the final rounding to fp32: each such row within 1e-6
relative error; the per-cell rows keep the extension's bar (1e-4 relative
Frobenius error over the chunk).  Cases: ranks 8 to 64, fixed tables below
and above 4 MiB (the two forms of the threshold), the step options and both
clip forms, rows just below and at the threshold, thresholds forced from the
environment (every row, none), chunking invariance, and thresholds that stay
off where the per-cell form is cheaper (k = 128, one step, k = 64 with a
table in L2).
"""
import os

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, rel_fro

pytestmark = pytest.mark.gpu

ROW_TOL = 1e-6
FP32_TOL = 1e-4


def _gram_min(k, steps, n_fixed):
    """The library's automatic threshold (extend_gram_min), restated: by
    arithmetic when the fixed table fits 4 MiB, else counting the per-cell
    form's gathers."""
    if k > 64 or steps < 1:
        return 0
    nb = (k + 15) // 16
    r = nb * (nb + 1) / 2 / (nb * nb)
    in_l2 = n_fixed * k * 4 <= 4 << 20
    den = (2.0 if in_l2 else 4.0) * steps - k * r
    if den <= 0:
        return 0
    return max(16, int(np.ceil(steps * k / den if in_l2 else 192.0 * steps / den)))


def _chunk(seed, k, n_fixed, lengths):
    """Free row f gets lengths[f] distinct cells (fixed ids drawn without
    repeats), shuffled; fixed factors of the scale the extension sees."""
    g = np.random.default_rng(seed)
    F = (g.standard_normal((n_fixed, k)) * k ** -0.5).astype(np.float32)
    fixed = np.concatenate([g.choice(n_fixed, n, replace=False) for n in lengths]).astype(np.int32)
    free = np.repeat(np.arange(len(lengths)), lengths).astype(np.int32)
    r = g.standard_normal(fixed.size).astype(np.float32)
    perm = g.permutation(fixed.size)
    return F, fixed[perm], free[perm], r[perm]


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    yield t
    t.close()


def _set_rank(T, k):
    p = synth.random_case(200, 150, 2000, 64, 48, k, seed=5)
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)


def _run(T, F, fixed, free, r, n_free, opts):
    import torch
    Fd = torch.from_numpy(F).cuda()
    out = torch.full((n_free, F.shape[1]), np.nan, dtype=torch.float32).pin_memory()
    T.extend_chunk(1, fixed, free, r, n_free, Fd, out, opts)
    T.sync()
    return out.numpy().copy()


def _row_err(X, Xo):
    num = np.linalg.norm(np.asarray(X, np.float64) - Xo, axis=1)
    den = np.linalg.norm(Xo, axis=1)
    return np.where(den > 0, num / np.maximum(den, 1e-300), num)


class _gram_env:
    """TSID_EXT_GRAM_MIN for the duration of a block (read at every chunk)."""

    def __init__(self, value):
        self.value = value

    def __enter__(self):
        self.old = os.environ.get("TSID_EXT_GRAM_MIN")
        os.environ["TSID_EXT_GRAM_MIN"] = str(self.value)

    def __exit__(self, *exc):
        if self.old is None:
            del os.environ["TSID_EXT_GRAM_MIN"]
        else:
            os.environ["TSID_EXT_GRAM_MIN"] = self.old


def _check(X, Xo, lengths, gmin):
    long_rows = np.asarray(lengths) >= gmin if gmin > 0 else np.zeros(len(lengths), bool)
    assert np.all(np.isfinite(X))
    assert rel_fro(X, Xo) <= FP32_TOL, rel_fro(X, Xo)
    if long_rows.any():
        err = _row_err(X[long_rows], Xo[long_rows])
        assert err.max() <= ROW_TOL, err.max()
    assert np.all(X[np.asarray(lengths) == 0] == 0.0)


@pytest.mark.parametrize("k,n_fixed", [(8, 2500), (16, 2500), (32, 2500), (32, 40000), (64, 20000)])
@pytest.mark.parametrize("step,clip", [("degree", False), ("sum", False), ("degree", True),
                                       ("degree", "printed")])
def test_gram_rows_match_oracle(T, k, n_fixed, step, clip):
    """Automatic threshold at 20 steps, with fixed tables below and above
    4 MiB: rows on both sides of it, one without cells, one far longer than
    the rest."""
    from paper_2608_00977_amd import make_opts
    steps, lam, lr, xi = 20, 0.05, 0.05 if step == "degree" else 0.002, 0.02
    gmin = _gram_min(k, steps, n_fixed)
    assert gmin > 0
    lengths = [0, 1, gmin - 1, gmin, gmin + 1, 3 * gmin, 2000] + list(range(2, 200, 7))
    F, fixed, free, r = _chunk(100 + k, k, n_fixed, lengths)
    _set_rank(T, k)
    note(f"gram rows k={k} {step} clip={clip} gram_min={gmin}")
    X = _run(T, F, fixed, free, r, len(lengths), make_opts(epochs=steps, lam=lam, lr=lr, step=step, clip=clip,
                                                            xi=xi))
    st, Xo = oracle.extend(fixed, free, r, len(lengths), F, steps, lam, lr, step, clip, xi)
    assert st == 0
    _check(X, Xo, lengths, gmin)


@pytest.mark.parametrize("k", [16, 32, 64])
def test_forced_thresholds_match_oracle(T, k):
    """Every row with at least one cell in Gram form (threshold 1), then none
    (threshold -1): both against the oracle, and the Gram rows within the
    tighter bar."""
    from paper_2608_00977_amd import make_opts
    steps, lam, lr = 20, 0.02, 0.05
    lengths = [0, 1, 3, 17, 64, 65, 300, 1200] + list(range(5, 400, 37))
    F, fixed, free, r = _chunk(200 + k, k, 3000, lengths)
    _set_rank(T, k)
    opts = make_opts(epochs=steps, lam=lam, lr=lr, step="degree")
    st, Xo = oracle.extend(fixed, free, r, len(lengths), F, steps, lam, lr, "degree")
    assert st == 0
    for forced in (1, -1):
        note(f"gram forced k={k} threshold={forced}")
        with _gram_env(forced):
            X = _run(T, F, fixed, free, r, len(lengths), opts)
        _check(X, Xo, lengths, 1 if forced > 0 else 0)


def test_gram_chunking_is_invariant(T):
    """Rows in three chunks in flight equal one chunk bit for bit (each row's
    form depends on its own length only)."""
    import torch
    from paper_2608_00977_amd import make_opts
    k, steps = 32, 20
    lengths = [0] + [int(x) for x in np.random.default_rng(7).integers(1, 400, 89)]
    F, fixed, free, r = _chunk(7, k, 2000, lengths)
    _set_rank(T, k)
    opts = make_opts(epochs=steps, lam=0.05, lr=0.05, step="degree", clip=True, xi=0.02)
    note("gram chunking")
    whole = _run(T, F, fixed, free, r, 90, opts)
    Fd = torch.from_numpy(F).cuda()
    outs = []
    for lo, hi in ((0, 30), (30, 61), (61, 90)):
        m = (free >= lo) & (free < hi)
        out = torch.empty((hi - lo, k), dtype=torch.float32).pin_memory()
        T.extend_chunk(1, fixed[m], (free[m] - lo).astype(np.int32), r[m], hi - lo, Fd, out, opts)
        outs.append(out)
    T.sync()
    assert np.array_equal(np.concatenate([o.numpy() for o in outs]), whole)
    assert (np.asarray(lengths) >= _gram_min(k, steps, 2000)).sum() > 10


def test_gram_off_where_per_cell_is_cheaper(T):
    """k = 128 and a single step keep the per-cell form (the automatic rule
    returns no threshold), and the results still match the oracle."""
    from paper_2608_00977_amd import make_opts
    assert _gram_min(128, 20, 10 ** 6) == 0 and _gram_min(32, 1, 10 ** 6) == 0
    assert _gram_min(64, 20, 1000) == 0 and _gram_min(64, 10, 10 ** 6) == 0
    lengths = [0, 5, 300, 900]
    for k, steps in ((128, 3), (32, 1)):
        F, fixed, free, r = _chunk(300 + k, k, 1000, lengths)
        _set_rank(T, k)
        note(f"gram off k={k} steps={steps}")
        X = _run(T, F, fixed, free, r, len(lengths), make_opts(epochs=steps, lam=0.05, lr=0.05, step="degree"))
        st, Xo = oracle.extend(fixed, free, r, len(lengths), F, steps, 0.05, 0.05, "degree")
        assert st == 0 and rel_fro(X, Xo) <= FP32_TOL


def test_nonfinite_reported_in_both_forms(T):
    """A non-finite value on a row in Gram form, then on a row in the
    per-cell form: the next sync reports E_NONFINITE either way, and a clean
    chunk afterwards matches the oracle again."""
    import torch
    from paper_2608_00977_amd import TsidError, make_opts
    from paper_2608_00977_amd.binding import E_NONFINITE
    k, steps = 32, 20
    gmin = _gram_min(k, steps, 2000)
    opts = make_opts(epochs=steps, lam=0.05, lr=0.05, step="degree")
    _set_rank(T, k)
    for form, length in (("gram", 3 * gmin), ("per cell", gmin // 2)):
        F, fixed, free, r = _chunk(11, k, 2000, [length, 5])
        r = r.copy()
        r[np.flatnonzero(free == 0)[1]] = np.nan
        Fd = torch.from_numpy(F).cuda()
        out = torch.empty((2, k), dtype=torch.float32).pin_memory()
        note(f"gram nonfinite: {form} row of {length} cells")
        T.extend_chunk(1, fixed, free, r, 2, Fd, out, opts)
        with pytest.raises(TsidError) as e:
            T.sync()
        assert e.value.status == E_NONFINITE
    lengths = [0, 4, 3 * gmin]
    F, fixed, free, r = _chunk(12, k, 2000, lengths)
    X = _run(T, F, fixed, free, r, len(lengths), opts)
    st, Xo = oracle.extend(fixed, free, r, len(lengths), F, steps, 0.05, 0.05, "degree")
    assert st == 0
    _check(X, Xo, lengths, gmin)
