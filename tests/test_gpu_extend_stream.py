"""The chunked extension streamed at the workloads that define it (Section
5.2: double-buffered pipelining of chunks from the host), through the C ABI.

* Scientific: the whole 200,000 x 200,000 matrix outside the 16,384 x 16,384
  template -- the row phase (free rows against the template columns, about
  3e8 cells) and the column phase (free columns against every row, about
  3.3e9 cells) -- in chunks of at most 2^28 cells, generated a chunk at a
  time into two pinned host buffers.
* Billion-scale: the 10 M x 1 M matrix outside the 1 M x 100 k template, its
  Omega (about 6e8 cells) in chunks of at most 2^26 cells and the 9 M
  non-template row factors of the row phase returned to the host; the column
  phase reads all 10 M row factors (5 GB fp32) from the device.

Parity on sampled outputs the oracle computes one by one: a free row's
result depends only on its own cells and the fixed factors, so the oracle
(or_extend, fp64) recomputes sampled free rows (and the longest ones) from
their cells and the template's column factors, and sampled free columns
from their cells and the row factors the library's row phase produced (each
phase is thereby checked on its own), within 1e-4 relative Frobenius error.
The tests also check that the phases' cell counts partition the matrix's
cells outside the template and that every chunk stays under its cap.
"""
import time

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, rel_fro

pytestmark = pytest.mark.gpu

STEPS, LR = 20, 0.05


def _fit_template(T, p, epochs):
    import torch
    from paper_2608_00977_amd import make_opts
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    P = torch.from_numpy(p.P0).cuda()
    Q = torch.from_numpy(p.Q0).cuda()
    T.fit_template(P, Q, make_opts(epochs=epochs, lam=p.lam, lr=p.lr, clip=p.clip, xi=p.xi, prec=p.prec,
                                   step=p.step), want_loss=False)
    return P, Q


def _sample(counts, n, seed):
    g = np.random.default_rng(seed)
    top = np.argsort(-counts, kind="stable")[:2]
    return np.union1d(g.choice(counts.size, n, replace=False), top)


def _check_lines(phase, lines, F_fixed, got, lam, what):
    """Oracle solves of the sampled free lines from their own cells."""
    fixed, fl, r = phase.cells(lines)
    uniq, inv = np.unique(fixed, return_inverse=True)  # only the fixed rows they touch
    pos = np.searchsorted(lines, fl)
    st, X = oracle.extend(inv.astype(np.int32), pos.astype(np.int32), r, lines.size,
                          np.asarray(F_fixed[uniq], np.float64), STEPS, lam, LR, "degree")
    assert st == 0
    err = rel_fro(got[lines], X)
    note(f"{what}: {lines.size} lines, {r.size} cells, rel err {err:.2e}")
    assert err <= 1e-4


def _run(T, p, omega, max_entries, n_sample):
    import torch
    from paper_2608_00977_amd import make_opts
    from paper_2608_00977_amd.extension import StreamedExtension
    t0 = time.perf_counter()
    rows, cols = omega.row_phase(), omega.col_phase()
    note(f"{p.name} stream: counted {rows.nnz} row-phase and {cols.nnz} column-phase cells "
         f"({time.perf_counter() - t0:.0f}s)")
    P_t, Q_t = _fit_template(T, p, 3)
    ext = StreamedExtension(p.m, p.n, p.I, p.J, rows, cols, max_entries)
    for ph, b in zip((rows, cols), ext.bounds):
        c = np.concatenate([[0], np.cumsum(ph.counts)])
        per = c[b[1:]] - c[b[:-1]]
        assert b[0] == 0 and b[-1] == ph.counts.size and np.all(np.diff(b) > 0)
        assert np.all((per <= max_entries) | (np.diff(b) == 1))
    note(f"{p.name} stream: {ext.bounds[0].size - 1} + {ext.bounds[1].size - 1} chunks")
    opts = make_opts(epochs=STEPS, lam=p.lam, lr=LR, step="degree")
    T.set_timing(1)
    t0 = time.perf_counter()
    P_full, P_free, Q_free, ph = ext.run(T, P_t, Q_t, opts)
    tm = T.timing()
    T.set_timing(0)
    note(f"{p.name} stream: {time.perf_counter() - t0:.1f}s {ph}; copies {tm['ext_h2d_ms']:.0f} ms, compute "
         f"{tm['ext_compute_ms']:.0f} ms over {tm['ext_chunks']} chunks")
    assert tm["ext_chunks"] == ext.bounds[0].size + ext.bounds[1].size - 2
    assert P_free.is_cuda and not Q_free.is_cuda  # the row phase's factors stay in HBM
    P_free = P_free.cpu()
    assert np.all(np.isfinite(P_free.numpy())) and np.all(np.isfinite(Q_free.numpy()))
    Qt = Q_t.cpu().numpy()
    _check_lines(rows, _sample(rows.counts, n_sample, 1), Qt, P_free.numpy(), p.lam, f"{p.name} row phase")
    Pf = P_full.cpu().numpy()
    _check_lines(cols, _sample(cols.counts, n_sample, 2), Pf, Q_free.numpy(), p.lam, f"{p.name} column phase")
    return rows, cols


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    yield t
    t.close()


@pytest.mark.timeout(900)
def test_scientific_extension_streamed_fullsize(T):
    p = synth.scientific_template()
    note(f"scientific stream: template {p.I.size} x {p.J.size}, {p.nnz} training cells")
    rows, cols = _run(T, p, synth.omega_outside_template(p), 1 << 28, 40)
    # every training cell outside the template block is in exactly one phase:
    # the row phase takes the free rows' template-column cells, the column
    # phase every free column's cells; about 10 % of the matrix is observed
    # and 90 % of that is for training
    total = rows.nnz + cols.nnz + p.nnz
    assert abs(total / (0.1 * 0.9 * p.m * p.n) - 1.0) < 1e-3


@pytest.mark.timeout(900)
def test_billion_extension_streamed_fullsize(T):
    p = synth.billion_template()
    note(f"billion stream: template {p.I.size} x {p.J.size}, {p.nnz} training cells")
    omega = synth.omega_outside_template(p)
    rows, cols = _run(T, p, omega, 1 << 26, 40)
    total = rows.nnz + cols.nnz + p.nnz
    note(f"billion stream: {total} training cells in all ({total / 0.9:.3e} observed)")
    assert abs(total / 0.9 / 1e9 - 1.0) < 0.05
