"""Shared helpers of the GPU tests: run a Problem through the HIP library and
through the oracle on the same seeded inputs."""
import sys

import numpy as np

import oracle


def note(msg: str):
    """Names the case on stdout before a GPU step (flushed)."""
    print(f"[case] {msg}", flush=True)
    sys.stdout.flush()


def oracle_template(p):
    st, rm, cm = oracle.template_maps(p.m, p.n, p.I, p.J)
    assert st == 0
    a, b, v = oracle.filter_template(p.u, p.i, p.r, rm, cm)
    return rm, cm, a, b, v


def rel_fro(x, ref):
    ref = np.asarray(ref, np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(np.asarray(x, np.float64) - ref) / (den if den > 0 else 1.0))


def gpu_fit(T, p, epochs=None, prec=None, clip=None, lr=None, step=None, P0=None, Q0=None):
    import torch
    from paper_2608_00977_amd import make_opts
    P = torch.from_numpy(np.ascontiguousarray(p.P0 if P0 is None else P0, np.float32)).cuda()
    Q = torch.from_numpy(np.ascontiguousarray(p.Q0 if Q0 is None else Q0, np.float32)).cuda()
    opts = make_opts(epochs=p.epochs if epochs is None else epochs, lam=p.lam,
                     lr=p.lr if lr is None else lr, clip=p.clip if clip is None else clip, xi=p.xi,
                     prec=p.prec if prec is None else prec, step=p.step if step is None else step)
    st, hist = T.fit_template(P, Q, opts, raise_on_error=False)
    return st, P.cpu().numpy(), Q.cpu().numpy(), hist


def rmse_on(T_test, P, Q, n_test):
    """Held-out RMSE from the library's loss on a template built over the test cells."""
    import torch
    Pt = torch.from_numpy(np.ascontiguousarray(P, np.float32)).cuda()
    Qt = torch.from_numpy(np.ascontiguousarray(Q, np.float32)).cuda()
    sse = T_test.loss(Pt, Qt, 0.0)
    return float(np.sqrt(sse / max(1, n_test)))


def oracle_rmse(P, Q, p):
    """Held-out RMSE of oracle factors, through the oracle's own filter and loss."""
    st, rm, cm = oracle.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle.filter_template(p.tu, p.ti, p.tr, rm, cm)
    sse = oracle.loss(a, b, v, P.shape[0], Q.shape[0], P, Q, 0.0)
    return float(np.sqrt(sse / max(1, a.size))), a.size
