"""Extension chunks (Section 5.2) against the oracle, chunking invariance, and
the documented error paths of the C ABI (GPU)."""
import numpy as np
import pytest

import oracle
import tsid_synth as synth
from gpu_util import gpu_fit, note, oracle_template, rel_fro

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_2608_00977_amd as tsid
    t = tsid.Tsid(0)
    p = synth.random_case(200, 150, 2000, 64, 48, 32, seed=5)
    t.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)  # sets k = 32
    yield t
    t.close()


def _chunk(seed, n_fixed, n_free, nnz, k, hot=0):
    g = np.random.default_rng(seed)
    F = g.normal(0, k ** -0.25, (n_fixed, k)).astype(np.float32)
    cells = g.choice(n_fixed * n_free, min(nnz, n_fixed * n_free), replace=False)
    if hot:
        extra = np.arange(n_fixed) * n_free + 3  # free row 3 fully observed
        cells = np.unique(np.concatenate([cells, extra]))
        cells = cells[g.permutation(cells.size)]
    fixed = (cells // n_free).astype(np.int32)
    free = (cells % n_free).astype(np.int32)
    r = g.standard_normal(cells.size).astype(np.float32)
    return F, fixed, free, r


def _run(T, F, fixed, free, r, n_free, opts):
    import torch
    Fd = torch.from_numpy(F).cuda()
    out = torch.empty((n_free, F.shape[1]), dtype=torch.float32).pin_memory()
    T.extend_chunk(1, fixed, free, r, n_free, Fd, out, opts)
    T.sync()
    return out.numpy().copy()


@pytest.mark.parametrize("step,clip", [("degree", False), ("sum", False), ("degree", True)])
def test_extend_chunk_matches_oracle(T, step, clip):
    from paper_2608_00977_amd import make_opts
    F, fixed, free, r = _chunk(1, 3000, 700, 40000, 32, hot=1)
    lr = 0.2 if step == "degree" else 0.01
    note(f"extend step={step} clip={clip}")
    opts = make_opts(epochs=15, lam=0.01, lr=lr, clip=clip, xi=0.05, step=step)
    X = _run(T, F, fixed, free, r, 700, opts)
    st, Xo = oracle.extend(fixed, free, r, 700, F, 15, 0.01, lr, step, clip, 0.05)
    assert st == 0
    assert rel_fro(X, Xo) <= 1e-4


def test_extend_converges_to_ridge_solution(T):
    """Many one-sided steps reach the exact ridge minimiser (normal equations
    solved by the oracle's Cholesky; itself pinned to numpy lstsq)."""
    from paper_2608_00977_amd import make_opts
    F, fixed, free, r = _chunk(2, 400, 50, 8000, 32)
    note("extend ridge")
    X = _run(T, F, fixed, free, r, 50, make_opts(epochs=3000, lam=0.5, lr=0.4, step="degree"))
    st, Xr = oracle.ridge(fixed, free, r, 50, F, 0.5)
    assert st == 0
    assert rel_fro(X, Xr) <= 1e-4


def test_extend_pipeline_chunking_is_invariant(T):
    """A free row's result does not depend on which chunk carries it: three
    chunks in flight (double-buffered) reproduce one big chunk bit for bit."""
    import torch
    from paper_2608_00977_amd import make_opts
    F, fixed, free, r = _chunk(3, 2000, 900, 60000, 32, hot=1)
    opts = make_opts(epochs=10, lam=0.01, lr=0.2, step="degree")
    note("extend chunking")
    whole = _run(T, F, fixed, free, r, 900, opts)
    Fd = torch.from_numpy(F).cuda()
    bounds = [0, 250, 251, 900]
    outs = []
    for lo, hi in zip(bounds[:-1], bounds[1:]):
        sel = (free >= lo) & (free < hi)
        out = torch.empty((hi - lo, 32), dtype=torch.float32).pin_memory()
        T.extend_chunk(1, fixed[sel].copy(), (free[sel] - lo).astype(np.int32), r[sel].copy(),
                       hi - lo, Fd, out, opts)
        outs.append(out)
    T.sync()
    got = np.concatenate([o.numpy() for o in outs])
    assert np.array_equal(got, whole)


def test_chunk_plan_matches_oracle():
    from paper_2608_00977_amd import tsid_chunk_plan
    g = np.random.default_rng(8)
    for _ in range(30):
        counts = g.integers(0, 40, int(g.integers(0, 80))) * (g.random(1) < 0.9)
        for K in (1, 4, 16):
            assert np.array_equal(tsid_chunk_plan(counts, n_chunks=K), oracle.chunk_plan(counts, K))
        assert np.array_equal(tsid_chunk_plan(counts, max_entries=55),
                              oracle.chunk_plan(counts, max_entries=55))


# ------------------------------------------------------------------ errors
def _status(fn):
    from paper_2608_00977_amd import TsidError
    try:
        fn()
    except TsidError as e:
        return e.status
    return 0


def test_build_errors_leave_template_unchanged():
    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.binding import E_DUP, E_INVAL, E_RANGE, E_STATE
    p = synth.random_case(50, 40, 300, 20, 15, 8, seed=9)
    T = tsid.Tsid(0)
    try:
        import torch
        P = torch.zeros((20, 8), device="cuda")
        Q = torch.zeros((15, 8), device="cuda")
        note("errors: fit before build")
        assert _status(lambda: T.fit_template(P, Q, tsid.make_opts())) == E_STATE
        T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, 8)
        before = T.info()
        bad_u = p.u.copy()
        bad_u[7] = p.m
        cases = {
            "u out of range": (lambda: T.build_template(p.m, p.n, bad_u, p.i, p.r, p.I, p.J, 8), E_RANGE),
            "I out of range": (lambda: T.build_template(p.m, p.n, p.u, p.i, p.r,
                                                        np.append(p.I[:-1], p.m), p.J, 8), E_RANGE),
            "I repeats": (lambda: T.build_template(p.m, p.n, p.u, p.i, p.r,
                                                   np.append(p.I[:-1], p.I[0]), p.J, 8), E_DUP),
            "k = 7": (lambda: T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, 7), E_INVAL),
        }
        rm = {int(x): 1 for x in p.I}
        cm = {int(x): 1 for x in p.J}
        inside = [e for e in range(p.nnz) if int(p.u[e]) in rm and int(p.i[e]) in cm]
        dup_u = np.append(p.u, p.u[inside[0]])
        dup_i = np.append(p.i, p.i[inside[0]])
        dup_r = np.append(p.r, np.float32(1.0))
        cases["repeated cell inside the template"] = (
            lambda: T.build_template(p.m, p.n, dup_u, dup_i, dup_r, p.I, p.J, 8), E_DUP)
        outside = [e for e in range(p.nnz) if not (int(p.u[e]) in rm and int(p.i[e]) in cm)]
        dup2_u = np.append(p.u, p.u[outside[0]])
        dup2_i = np.append(p.i, p.i[outside[0]])
        dup2_r = np.append(p.r, np.float32(2.0))
        cases["repeated cell outside the template"] = (
            lambda: T.build_template(p.m, p.n, dup2_u, dup2_i, dup2_r, p.I, p.J, 8), E_DUP)
        cases["repeated cell outside the template, small staging pieces"] = (
            lambda: T.build_template(p.m, p.n, dup2_u, dup2_i, dup2_r, p.I, p.J, 8, stage_entries=37), E_DUP)
        nan_r = p.r.copy()
        nan_r[inside[1]] = np.nan
        cases["NaN value inside the template"] = (
            lambda: T.build_template(p.m, p.n, p.u, p.i, nan_r, p.I, p.J, 8), E_INVAL)
        for what, (fn, want) in cases.items():
            note(f"errors: {what}")
            assert _status(fn) == want, what
            assert T.info() == before, what
    finally:
        T.close()


def test_nonfinite_returns_last_finite_iterate(T):
    p = synth.random_case(200, 150, 2000, 64, 48, 32, seed=5, step="sum")
    T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, p.k)
    from paper_2608_00977_amd.binding import E_NONFINITE
    note("errors: non-finite")
    st, P, Q, hist = gpu_fit(T, p, epochs=60, lr=50.0, step="sum")
    assert st == E_NONFINITE
    done = T.epochs_done()
    assert 0 < done < 60 and np.all(np.isfinite(P)) and np.all(np.isfinite(Q))
    assert np.all(np.isnan(hist[done + 1:]))
    st2, P2, Q2, h2 = gpu_fit(T, p, epochs=done, lr=50.0, step="sum")
    assert st2 == 0 and T.epochs_done() == done
    assert np.array_equal(P, P2) and np.array_equal(Q, Q2)
    # the oracle (fp64) also leaves the finite range, later: fp32 overflows first
    _, _, a, b, v = oracle_template(p)
    sto, _, _, _, done_o = oracle.fit(a, b, v, p.P0, p.Q0, 60, p.lam, 50.0, "sum")
    assert sto == 7 and done_o >= done


def test_extension_device_errors_reported_by_sync(T):
    import torch
    from paper_2608_00977_amd import make_opts
    from paper_2608_00977_amd.binding import E_DUP, E_RANGE
    F, fixed, free, r = _chunk(4, 100, 30, 500, 32)
    Fd = torch.from_numpy(F).cuda()
    out = torch.empty((30, 32), dtype=torch.float32).pin_memory()
    opts = make_opts(epochs=2, lam=0.01, lr=0.1, step="degree")
    bad = fixed.copy()
    bad[3] = 100
    note("errors: extension range")
    T.extend_chunk(1, bad, free, r, 30, Fd, out, opts)
    assert _status(T.sync) == E_RANGE
    note("errors: extension duplicate")
    T.extend_chunk(1, np.append(fixed, fixed[0]), np.append(free, free[0]), np.append(r, r[0]), 30,
                   Fd, out, opts)
    assert _status(T.sync) == E_DUP
    T.extend_chunk(1, fixed, free, r, 30, Fd, out, opts)
    T.sync()  # clean again


def test_bad_device_id():
    """tsid_create with a device id the runtime does not have: E_DEVICE."""
    import torch
    from paper_2608_00977_amd.binding import E_DEVICE, TsidError, tsid_create
    with pytest.raises(TsidError) as ei:
        tsid_create(torch.cuda.device_count(), 0, 0)
    assert ei.value.status == E_DEVICE


def test_device_byte_cap():
    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.binding import E_NOMEM
    p = synth.random_case(400, 300, 5000, 100, 80, 32, seed=3)
    T = tsid.Tsid(0, max_device_bytes=64 * 1024)
    try:
        note("errors: byte cap")
        assert _status(lambda: T.build_template(p.m, p.n, p.u, p.i, p.r, p.I, p.J, 32)) == E_NOMEM
    finally:
        T.close()


@pytest.mark.parametrize("n_fixed,n_free", [(200, 200), (3000, 700), (3000, 5000), (1 << 20, 5000)])
def test_sorted_chunk_skips_the_sort_same_bits(T, n_fixed, n_free):
    """A chunk already in (free row, fixed id) order skips the radix passes;
    its result equals the shuffled chunk's bit for bit, with the key widths
    giving 2, 3, 4 and 5 passes (an odd count leaves the sorted keys in the
    other buffer), and matches the oracle."""
    from paper_2608_00977_amd import make_opts
    k = 32
    g = np.random.default_rng(n_fixed + n_free)
    nnz = min(30000, n_fixed * n_free // 4)
    cells = g.choice(n_fixed * n_free, nnz, replace=False)
    F = g.normal(0, k ** -0.25, (n_fixed, k)).astype(np.float32)
    fixed = (cells % n_fixed).astype(np.int32)
    free = (cells // n_fixed).astype(np.int32)
    r = g.standard_normal(nnz).astype(np.float32)
    order = np.lexsort((fixed, free))
    opts = make_opts(epochs=10, lam=0.01, lr=0.1, step="degree")
    note(f"sorted chunk n_fixed={n_fixed} n_free={n_free}")
    X_shuffled = _run(T, F, fixed, free, r, n_free, opts)
    X_sorted = _run(T, F, fixed[order], free[order], r[order], n_free, opts)
    assert np.array_equal(X_sorted, X_shuffled)
    st, Xo = oracle.extend(fixed, free, r, n_free, F, 10, 0.01, 0.1, "degree")
    assert st == 0
    assert rel_fro(X_sorted, Xo) <= 1e-4


def test_sorted_chunk_with_a_repeat_reports_duplicate(T):
    import torch
    from paper_2608_00977_amd import make_opts
    from paper_2608_00977_amd.binding import E_DUP
    F, fixed, free, r = _chunk(4, 100, 30, 500, 32)
    order = np.lexsort((fixed, free))
    fixed, free, r = fixed[order], free[order], r[order]
    j = 7  # repeat cell j right after it: the keys stay in order
    fixed = np.insert(fixed, j + 1, fixed[j])
    free = np.insert(free, j + 1, free[j])
    r = np.insert(r, j + 1, r[j])
    Fd = torch.from_numpy(F).cuda()
    out = torch.empty((30, 32), dtype=torch.float32).pin_memory()
    note("errors: duplicate in a sorted chunk")
    T.extend_chunk(1, fixed, free, r, 30, Fd, out, make_opts(epochs=2, lam=0.01, lr=0.1, step="degree"))
    assert _status(T.sync) == E_DUP


def test_device_output_equals_host_output(T):
    """F_free in device memory receives the same bits as a pinned host buffer
    (the results are copied on the device), for the steps and the exact solve."""
    import torch
    from paper_2608_00977_amd import make_opts
    F, fixed, free, r = _chunk(31, 3000, 700, 40000, 32, hot=1)
    Fd = torch.from_numpy(F).cuda()
    for opts in (make_opts(epochs=15, lam=0.01, lr=0.2, step="degree"), 0.05):
        note(f"device output {'steps' if not isinstance(opts, float) else 'ridge'}")
        host = torch.empty((700, 32), dtype=torch.float32).pin_memory()
        dev = torch.full((700, 32), float("nan"), dtype=torch.float32, device="cuda")
        T.extend_chunk(1, fixed, free, r, 700, Fd, host, opts)
        T.extend_chunk(1, fixed, free, r, 700, Fd, dev, opts)
        T.sync()
        assert np.array_equal(dev.cpu().numpy(), host.numpy())
