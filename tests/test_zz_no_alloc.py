"""tsid_loss_noalloc (the allocation-free variant of tsid_loss) through the
C ABI: the same value as tsid_loss, bit for bit, on two calls in a row, the
second on a smaller template (the scratch array still holds the first
call's larger contents), also from a second context on the same device; a
template beyond the scratch limit is rejected with E_NOMEM before any
launch.  tsid_loss itself is checked against the oracle's Eq. 2 elsewhere;
here both are also compared with it at the loss bar (1e-6)."""
import ctypes as C

import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import note, oracle_template

pytestmark = pytest.mark.gpu


def _factors(p, seed):
    g = synth.make_rng(seed, "init")
    return (g.normal(0.0, 0.5, (p.I.size, p.k)).astype(np.float32),
            g.normal(0.0, 0.5, (p.J.size, p.k)).astype(np.float32))


def _both(T, p, lam, seed):
    import torch
    from paper_2608_00977_amd.binding import _ptr, tsid_loss, tsid_loss_noalloc
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    Pn, Qn = _factors(p, seed)
    P, Q = torch.from_numpy(Pn).cuda(), torch.from_numpy(Qn).cuda()
    torch.cuda.synchronize()
    ref = np.zeros(1, np.float64)
    got = np.zeros(1, np.float64)
    assert tsid_loss(T.ctx, _ptr(P), _ptr(Q), lam, _ptr(ref)) == 0
    assert tsid_loss_noalloc(T.ctx, _ptr(P), _ptr(Q), lam, _ptr(got)) == 0
    _, _, a, b, v = oracle_template(p)
    want = oracle.loss(a, b, v, p.I.size, p.J.size, Pn, Qn, lam)
    return float(ref[0]), float(got[0]), want


def test_noalloc_loss_equals_loss_twice_then_smaller():
    import paper_2608_00977_amd as tsid
    T = tsid.Tsid(0)
    T2 = tsid.Tsid(0)
    try:
        big = synth.mid()
        note(f"noalloc loss: mid m_t={big.I.size} n_t={big.J.size} nnz={big.nnz}")
        ref, got, want = _both(T, big, 1e-3, 1)
        assert got == ref, (got, ref)
        assert abs(got - want) <= 1e-6 * abs(want)
        small = synth.tiny()
        note(f"noalloc loss: tiny m_t={small.I.size} n_t={small.J.size} nnz={small.nnz}")
        ref, got, want = _both(T, small, 0.5, 2)
        assert got == ref, (got, ref)
        assert abs(got - want) <= 1e-6 * abs(want)
        # another context on the same device shares the array (sequential calls)
        rc = synth.random_case(700, 500, 9000, 300, 200, 32, seed=11, hot_rows=3, hot_cols=2)
        note("noalloc loss: second context")
        ref, got, want = _both(T2, rc, 0.0, 3)
        assert got == ref, (got, ref)
        assert abs(got - want) <= 1e-6 * abs(want)
    finally:
        T.close()
        T2.close()


def test_noalloc_loss_rejects_a_template_beyond_the_scratch():
    import torch
    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.binding import _ptr, tsid_loss_noalloc
    T = tsid.Tsid(0)
    try:
        # 4.5 M template rows: at least one work item and one norm per row,
        # 36 MB of scratch against 32 MiB
        m_t, n = 4_500_000, 64
        I = np.arange(m_t, dtype=np.int32)
        J = np.arange(n, dtype=np.int32)
        u = np.array([0, 1], np.int32)
        i = np.array([0, 1], np.int32)
        r = np.array([1.0, 2.0], np.float32)
        note("noalloc loss: over-limit template")
        T.build_template(m_t, n, u, i, r, I, J, 8)
        P = torch.zeros((m_t, 8), dtype=torch.float32, device="cuda")
        Q = torch.zeros((n, 8), dtype=torch.float32, device="cuda")
        out = np.full(1, -1.0)
        st = tsid_loss_noalloc(T.ctx, _ptr(P), _ptr(Q), 0.0, _ptr(out))
        assert st == 4  # TSID_E_NOMEM
        assert out[0] == -1.0
        assert "scratch" in tsid.binding.tsid_last_error(T.ctx)
        # the context stays usable
        assert T.loss(P, Q, 0.0) == pytest.approx(5.0)
    finally:
        T.close()
