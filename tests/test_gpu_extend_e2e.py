"""End-to-end extension (row phase, then column phase) on a scaled-down
Rating-shaped matrix, through the package's chunk driver and the C ABI,
against the oracle run on the same cells (GPU).

Both sides start from the same seeded template factors, so no oracle input
comes from the HIP path; the oracle's column phase uses the oracle's own
row-phase result."""
import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, rel_fro

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _oracle_phases(p, steps, lam, lr, step):
    """The two phases written out with numpy masks (independent of the
    package's driver), each as one oracle extension over all its cells."""
    u = p.u.astype(np.int64)
    i = p.i.astype(np.int64)
    row_in = np.zeros(p.m, bool)
    row_in[p.I] = True
    col_in = np.zeros(p.n, bool)
    col_in[p.J] = True
    cm = np.full(p.n, -1, np.int64)
    cm[p.J] = np.arange(p.J.size)
    F_rows = np.flatnonzero(~row_in)
    pos_r = np.full(p.m, -1, np.int64)
    pos_r[F_rows] = np.arange(F_rows.size)
    sel = ~row_in[u] & col_in[i]
    st, Xr = oracle.extend(cm[i[sel]], pos_r[u[sel]], p.r[sel], F_rows.size, p.Q0, steps, lam, lr,
                           step)
    assert st == 0
    P_full = np.zeros((p.m, p.k))
    P_full[p.I] = p.P0
    P_full[F_rows] = Xr
    F_cols = np.flatnonzero(~col_in)
    pos_c = np.full(p.n, -1, np.int64)
    pos_c[F_cols] = np.arange(F_cols.size)
    sel2 = ~col_in[i]
    st, Xc = oracle.extend(u[sel2], pos_c[i[sel2]], p.r[sel2], F_cols.size, P_full, steps, lam,
                           lr, step)
    assert st == 0
    used = int(sel.sum() + sel2.sum() + np.count_nonzero(row_in[u] & col_in[i]))
    return F_rows, Xr, F_cols, Xc, used


@pytest.mark.parametrize("n_chunks", [16, 3])
def test_extension_end_to_end_matches_oracle(n_chunks):
    import torch

    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.extension import Extension
    p = synth.rating(scale=0.05)
    steps, lam, lr, step = 12, 1e-3, 0.05, "degree"
    note(f"extension e2e rating(0.05) nnz={p.nnz} chunks={n_chunks}")
    T = tsid.Tsid(0)
    try:
        T.build_template(p.m, p.n, p.u[:0], p.i[:0], p.r[:0], p.I, p.J, p.k)  # sets k
        ext = Extension(p.m, p.n, p.u, p.i, p.r, p.I, p.J, n_chunks=n_chunks)
        assert ext.rows.bounds.size - 1 <= n_chunks and ext.cols.bounds.size - 1 <= n_chunks
        P_t = torch.from_numpy(p.P0).cuda()
        Q_t = torch.from_numpy(p.Q0).cuda()
        opts = tsid.make_opts(epochs=steps, lam=lam, lr=lr, step=step)
        P, Q, _ = ext.run(T, P_t, Q_t, opts)
    finally:
        T.close()
    P, Q = P.numpy(), Q.numpy()
    F_rows, Xr, F_cols, Xc, used = _oracle_phases(p, steps, lam, lr, step)
    # every training cell is used exactly once: template, row phase or column phase
    assert ext.rows.nnz + ext.cols.nnz + ext.template_nnz == p.nnz == used
    assert np.array_equal(P[p.I], p.P0) and np.array_equal(Q[p.J], p.Q0)
    assert rel_fro(P[F_rows], Xr) <= TOL, rel_fro(P[F_rows], Xr)
    assert rel_fro(Q[F_cols], Xc) <= TOL, rel_fro(Q[F_cols], Xc)


@pytest.mark.timeout(900)
def test_extension_fullsize_sampled_rating():
    """The full Rating-shaped extension (480,189 x 17,770, 100 M cells, 16
    chunks per phase, 20 one-sided steps: the bench.py --extend setting),
    checked on sampled outputs the oracle computes one by one: 64 free rows
    (plus the two with the most cells) from their template-column cells, and
    64 free columns (plus the two longest) from all their cells, with the
    row factors of the rows they touch taken from the oracle's own row phase
    of those rows."""
    import torch

    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.extension import Extension
    p = synth.rating()
    steps, lam, lr, step = 20, p.lam, 0.05, "degree"
    note(f"extension fullsize rating nnz={p.nnz}")
    T = tsid.Tsid(0)
    try:
        T.build_template(p.m, p.n, p.u[:0], p.i[:0], p.r[:0], p.I, p.J, p.k)  # sets k
        ext = Extension(p.m, p.n, p.u, p.i, p.r, p.I, p.J, n_chunks=16)
        opts = tsid.make_opts(epochs=steps, lam=lam, lr=lr, step=step)
        P, Q, _ = ext.run(T, torch.from_numpy(p.P0).cuda(), torch.from_numpy(p.Q0).cuda(), opts)
    finally:
        T.close()
    P, Q = P.numpy(), Q.numpy()
    u = p.u.astype(np.int64)
    i = p.i.astype(np.int64)
    row_in = np.zeros(p.m, bool)
    row_in[p.I] = True
    col_in = np.zeros(p.n, bool)
    col_in[p.J] = True
    cm = np.full(p.n, -1, np.int64)
    cm[p.J] = np.arange(p.J.size)
    in_tc = col_in[i]  # cells in template columns

    def row_phase(rows):
        """Oracle row phase of the given free rows (ascending global ids)."""
        pos = np.full(p.m, -1, np.int64)
        pos[rows] = np.arange(rows.size)
        sel = in_tc & (pos[u] >= 0)
        st, X = oracle.extend(cm[i[sel]], pos[u[sel]], p.r[sel], rows.size, p.Q0, steps, lam, lr,
                              step)
        assert st == 0
        return X

    g = np.random.default_rng(7)
    F_rows = np.flatnonzero(~row_in)
    cnt_r = np.bincount(u[in_tc & ~row_in[u]], minlength=p.m)[F_rows]
    rows = np.union1d(g.choice(F_rows, 64, replace=False), F_rows[np.argsort(-cnt_r, kind="stable")[:2]])
    assert rel_fro(P[rows], row_phase(rows)) <= TOL

    F_cols = np.flatnonzero(~col_in)
    cnt_c = np.bincount(i[~col_in[i]], minlength=p.n)[F_cols]
    cols = np.union1d(g.choice(F_cols, 64, replace=False), F_cols[np.argsort(-cnt_c, kind="stable")[:2]])
    posc = np.full(p.n, -1, np.int64)
    posc[cols] = np.arange(cols.size)
    sel = posc[i] >= 0
    touched = np.unique(u[sel])
    free_t = touched[~row_in[touched]]
    # row factors of the touched rows: template rows from P0, free rows from the oracle
    Psub = np.zeros((touched.size, p.k))
    tpos = np.full(p.m, -1, np.int64)
    tpos[p.I] = np.arange(p.I.size)
    is_t = row_in[touched]
    Psub[is_t] = p.P0[tpos[touched[is_t]]]
    Psub[~is_t] = row_phase(free_t)
    idx = np.full(p.m, -1, np.int64)
    idx[touched] = np.arange(touched.size)
    note(f"extension fullsize: {cols.size} columns over {touched.size} rows ({free_t.size} free)")
    st, Xc = oracle.extend(idx[u[sel]], posc[i[sel]], p.r[sel], cols.size, Psub, steps, lam, lr, step)
    assert st == 0
    assert rel_fro(Q[cols], Xc) <= TOL
