"""ctypes wrapper of the fp64 CPU oracle (``oracle/tsid_oracle.c``).

TEST INFRASTRUCTURE ONLY.  Import it from the tests, the smoke check or the
benchmark's CPU-baseline leg, never from the product package.  It shares no
code with the HIP path: it compiles its own C file with gcc.

Each wrapper converts its arguments with numpy and calls the C routine of the
same name (prefix ``or_``); the C header states which passage of the paper
each routine follows.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tsid_oracle.c")
_LIB = os.path.join(_HERE, "libtsid_oracle.so")
_LIB_OMP = os.path.join(_HERE, "libtsid_oracle_omp.so")


def _compile(out: str, extra) -> None:
    tmp = out + ".tmp%d" % os.getpid()
    subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-Wall", "-Wextra", "-Wno-unknown-pragmas", *extra, _SRC, "-o", tmp, "-lm"])
    os.replace(tmp, out)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain -O2, IEEE semantics, no FMA
    contraction): the serial library, and the same source with OpenMP (its
    parallel loops are those of or_fit_lines and a few elementwise copies)."""
    for out, extra in ((_LIB, []), (_LIB_OMP, ["-fopenmp"])):
        if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
            _compile(out, extra)
    return _LIB


_lib: Optional[C.CDLL] = None
_lib_omp: Optional[C.CDLL] = None


def lib(omp: bool = False) -> C.CDLL:
    """The serial oracle library, or (omp=True) the same source built with
    OpenMP (threads from OMP_NUM_THREADS, else all cores)."""
    global _lib, _lib_omp
    if omp:
        if _lib_omp is None:
            build(force=False)
            _lib_omp = _declare(C.CDLL(_LIB_OMP))
        return _lib_omp
    if _lib is None:
        _lib = _declare(C.CDLL(build(force=False)))
    return _lib


def _declare(lb: C.CDLL) -> C.CDLL:
    if True:  # signatures of the exported routines
        P = C.c_void_p
        i32, i64, f64 = C.c_int32, C.c_int64, C.c_double
        sig = {
            "or_template_maps": (C.c_int, [i64, i64, P, i32, P, i32, P, P]),
            "or_check_omega": (C.c_int, [i64, i64, i64, P, P, P]),
            "or_filter": (i64, [i64, P, P, P, P, P, P, P, P]),
            "or_bucket": (None, [i64, P, P, P, i32, i32, P, P, P, P, P, P, P, P]),
            "or_loss": (f64, [i64, P, P, P, i32, i32, i32, P, P, f64]),
            "or_fit": (C.c_int, [i64, P, P, P, i32, i32, i32, P, P, i32, f64, f64, i32, i32, f64,
                                 i32, P, P]),
            "or_extend": (C.c_int, [i64, P, P, P, i32, i32, P, P, i32, f64, f64, i32, i32, f64]),
            "or_ridge": (C.c_int, [i64, P, P, P, i32, i32, P, f64, P]),
            "or_splitmix64": (C.c_uint64, [C.c_uint64]),
            "or_batch_of": (i32, [i32, i32, C.c_uint64, i32]),
            "or_batch_of_many": (None, [i64, P, P, C.c_uint64, i32, P]),
            "or_fit_minibatch": (C.c_int, [i64, P, P, P, i32, i32, i32, P, P, i32, f64, f64, i32, i32,
                                           f64, i32, i32, C.c_uint64, P, P]),
            "or_extend_adam": (C.c_int, [i64, P, P, P, i32, i32, P, i32, P, i32, f64, f64, f64, f64,
                                         f64, P, P]),
            "or_chunk_plan": (i32, [P, i64, i32, i64, P, i32]),
            "or_loss_mv": (f64, [i64, P, P, P, i32, i32, i32, P, P, f64, i64, P, P, P, f64]),
            "or_fit_mv": (C.c_int, [i64, P, P, P, i32, i32, i32, P, P, i32, f64, f64, i32, i32, f64, i32,
                                    i64, P, P, P, f64, P, P]),
            "or_similarity": (None, [i32, i32, P, P]),
            "or_bf16_bits": (C.c_uint16, [C.c_float]),
            "or_fit_lines": (C.c_int, [i64, P, P, P, i32, i32, i32, P, P, i32, f64, f64, i32, i32, f64,
                                       i32, P, P]),
            "or_threads": (C.c_int, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lb, name)
            fn.restype = res
            fn.argtypes = args
    return lb


def _p(x: np.ndarray):
    return x.ctypes.data_as(C.c_void_p)


def _c(x, dtype):
    return np.ascontiguousarray(x, dtype=dtype)


STEP = {"sum": 0, "degree": 1, "col_degree": 2}
# clip option: False / True (1, on the normalised direction), "per_entry" (2),
# "printed" (3, on the summed direction before the step normalisation)
CLIP = {False: 0, True: 1, 0: 0, 1: 1, 2: 2, 3: 3, "per_entry": 2, "printed": 3}


def template_maps(m, n, I, J):
    I = _c(I, np.int32)
    J = _c(J, np.int32)
    rm = np.empty(m, np.int32)
    cm = np.empty(n, np.int32)
    st = lib().or_template_maps(m, n, _p(I), I.size, _p(J), J.size, _p(rm), _p(cm))
    return st, rm, cm


def check_omega(m, n, u, i, r) -> int:
    u, i, r = _c(u, np.int32), _c(i, np.int32), _c(r, np.float32)
    return lib().or_check_omega(m, n, u.size, _p(u), _p(i), _p(r))


def filter_template(u, i, r, row_map, col_map):
    u, i, r = _c(u, np.int32), _c(i, np.int32), _c(r, np.float32)
    rm, cm = _c(row_map, np.int32), _c(col_map, np.int32)
    a = np.empty(u.size, np.int32)
    b = np.empty(u.size, np.int32)
    v = np.empty(u.size, np.float32)
    cnt = lib().or_filter(u.size, _p(u), _p(i), _p(r), _p(rm), _p(cm), _p(a), _p(b), _p(v))
    return a[:cnt].copy(), b[:cnt].copy(), v[:cnt].copy()


def bucket(a, b, v, m_t, n_t) -> dict:
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    nnz = a.size
    out = dict(row_ptr=np.empty(m_t + 1, np.int64), csr_col=np.empty(nnz, np.int32),
               csr_val=np.empty(nnz, np.float32), col_ptr=np.empty(n_t + 1, np.int64),
               csc_row=np.empty(nnz, np.int32), csc_val=np.empty(nnz, np.float32),
               deg_r=np.empty(m_t, np.int32), deg_c=np.empty(n_t, np.int32))
    lib().or_bucket(nnz, _p(a), _p(b), _p(v), m_t, n_t, *[_p(out[k]) for k in
                    ("row_ptr", "csr_col", "csr_val", "col_ptr", "csc_row", "csc_val",
                     "deg_r", "deg_c")])
    return out


def loss(a, b, v, m_t, n_t, P, Q, lam) -> float:
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    P, Q = _c(P, np.float64), _c(Q, np.float64)
    return lib().or_loss(a.size, _p(a), _p(b), _p(v), m_t, n_t, P.shape[1], _p(P), _p(Q), lam)


def fit(a, b, v, P0, Q0, epochs, lam, lr, step="sum", clip=False, xi=0.1, bf16=False):
    """Returns (status, P, Q, loss_hist, epochs_done); P, Q are fp64."""
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    P = np.array(P0, dtype=np.float64, order="C", copy=True)
    Q = np.array(Q0, dtype=np.float64, order="C", copy=True)
    hist = np.full(epochs + 1, np.nan)
    done = np.zeros(1, np.int32)
    st = lib().or_fit(a.size, _p(a), _p(b), _p(v), P.shape[0], Q.shape[0], P.shape[1], _p(P),
                      _p(Q), epochs, lam, lr, STEP[step], CLIP[clip], xi, int(bf16), _p(hist),
                      _p(done))
    return st, P, Q, hist, int(done[0])


def fit_lines(a, b, v, P0, Q0, epochs, lam, lr, step="sum", clip=False, xi=0.1, bf16=False, omp=True):
    """or_fit_lines: the same result as fit(), bit for bit, with the rows and
    then the columns split across OpenMP threads (omp=True) or run serially.
    Returns (status, P, Q, loss_hist, epochs_done)."""
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    P = np.array(P0, dtype=np.float64, order="C", copy=True)
    Q = np.array(Q0, dtype=np.float64, order="C", copy=True)
    hist = np.full(epochs + 1, np.nan)
    done = np.zeros(1, np.int32)
    st = lib(omp).or_fit_lines(a.size, _p(a), _p(b), _p(v), P.shape[0], Q.shape[0], P.shape[1], _p(P), _p(Q),
                               epochs, lam, lr, STEP[step], CLIP[clip], xi, int(bf16), _p(hist), _p(done))
    return st, P, Q, hist, int(done[0])


def threads(omp: bool = True) -> int:
    """Threads the OpenMP build runs with (1 for the serial library)."""
    return int(lib(omp).or_threads())


def loss_mv(a, b, v, m_t, n_t, P, Q, lam, s_row, s_col, s_val, beta) -> float:
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    P, Q = _c(P, np.float64), _c(Q, np.float64)
    s_row, s_col, s_val = _c(s_row, np.int32), _c(s_col, np.int32), _c(s_val, np.float32)
    return lib().or_loss_mv(a.size, _p(a), _p(b), _p(v), m_t, n_t, P.shape[1], _p(P), _p(Q), lam, s_val.size,
                            _p(s_row), _p(s_col), _p(s_val), beta)


def fit_mv(a, b, v, P0, Q0, epochs, lam, lr, s_row, s_col, s_val, beta, step="sum", clip=False, xi=0.1,
           bf16=False):
    """The fit with the multi-view similarity term; returns as fit()."""
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    s_row, s_col, s_val = _c(s_row, np.int32), _c(s_col, np.int32), _c(s_val, np.float32)
    P = np.array(P0, np.float64, order="C", copy=True)
    Q = np.array(Q0, np.float64, order="C", copy=True)
    hist = np.full(epochs + 1, np.nan)
    done = np.zeros(1, np.int32)
    st = lib().or_fit_mv(a.size, _p(a), _p(b), _p(v), P.shape[0], Q.shape[0], P.shape[1], _p(P), _p(Q), epochs,
                         lam, lr, STEP[step], CLIP[clip], xi, int(bf16), s_val.size, _p(s_row), _p(s_col),
                         _p(s_val), beta, _p(hist), _p(done))
    return st, P, Q, hist, int(done[0])


def similarity(attr) -> np.ndarray:
    """Dense item similarity from categorical attributes (n x n_attr int)."""
    attr = _c(attr, np.int32)
    n, na = attr.shape
    S = np.zeros((n, n), np.float64)
    lib().or_similarity(n, na, _p(attr), _p(S))
    return S


def splitmix64(x: int) -> int:
    return int(lib().or_splitmix64(C.c_uint64(x & 0xFFFFFFFFFFFFFFFF)))


def batch_of(a: int, b: int, seed: int, n_batches: int) -> int:
    return int(lib().or_batch_of(int(a), int(b), C.c_uint64(seed), int(n_batches)))


def batch_of_many(a, b, seed: int, n_batches: int) -> np.ndarray:
    a, b = _c(a, np.int32), _c(b, np.int32)
    out = np.empty(a.size, np.int32)
    lib().or_batch_of_many(a.size, _p(a), _p(b), C.c_uint64(seed), int(n_batches), _p(out))
    return out


def fit_minibatch(a, b, v, P0, Q0, epochs, lam, lr, step="sum", clip=False, xi=0.1, bf16=False,
                  n_batches=2, seed=0):
    a, b, v = _c(a, np.int32), _c(b, np.int32), _c(v, np.float32)
    P = np.array(P0, np.float64, order="C", copy=True)
    Q = np.array(Q0, np.float64, order="C", copy=True)
    hist = np.full(epochs + 1, np.nan)
    done = np.zeros(1, np.int32)
    st = lib().or_fit_minibatch(a.size, _p(a), _p(b), _p(v), P.shape[0], Q.shape[0], P.shape[1], _p(P),
                                _p(Q), epochs, lam, lr, STEP[step], CLIP[clip], xi, int(bf16), n_batches,
                                C.c_uint64(seed), _p(hist), _p(done))
    return st, P, Q, hist, int(done[0])


def extend(fixed_id, free_id, v, n_free, F_fixed, steps, lam, lr, step="degree", clip=False,
           xi=0.1):
    fixed_id, free_id, v = _c(fixed_id, np.int32), _c(free_id, np.int32), _c(v, np.float32)
    F = _c(F_fixed, np.float64)
    k = F.shape[1]
    X = np.zeros((n_free, k), np.float64)
    st = lib().or_extend(v.size, _p(fixed_id), _p(free_id), _p(v), n_free, k, _p(F), _p(X),
                         steps, lam, lr, STEP[step], CLIP[clip], xi)
    return st, X


def ridge(fixed_id, free_id, v, n_free, F_fixed, lam):
    fixed_id, free_id, v = _c(fixed_id, np.int32), _c(free_id, np.int32), _c(v, np.float32)
    F = _c(F_fixed, np.float64)
    k = F.shape[1]
    X = np.zeros((n_free, k), np.float64)
    st = lib().or_ridge(v.size, _p(fixed_id), _p(free_id), _p(v), n_free, k, _p(F), lam, _p(X))
    return st, X


def extend_adam(fixed_id, free_id, v, n_free, F_fixed, B, steps, lam, lr, beta1=0.9, beta2=0.999,
                eps=1e-8):
    """Stage II as Eq. 6 states it (Section 5.2): Adam on the coefficients C of
    each free line in the template basis B.  Returns (status, B^T C per free
    line (n_free x k), C (n_free x n_b))."""
    fixed_id, free_id, v = _c(fixed_id, np.int32), _c(free_id, np.int32), _c(v, np.float32)
    F = _c(F_fixed, np.float64)
    Bm = _c(B, np.float64)
    k, n_b = F.shape[1], Bm.shape[0]
    X = np.zeros((n_free, k), np.float64)
    Cm = np.zeros((n_free, n_b), np.float64)
    st = lib().or_extend_adam(v.size, _p(fixed_id), _p(free_id), _p(v), n_free, k, _p(F), n_b, _p(Bm),
                              steps, lam, lr, beta1, beta2, eps, _p(X), _p(Cm))
    return st, X, Cm


def chunk_plan(counts, n_chunks=0, max_entries=0):
    counts = _c(counts, np.int64)
    cap = (n_chunks + 1) if n_chunks > 0 else counts.size + 2
    bounds = np.empty(max(cap, 2), np.int64)
    nc = lib().or_chunk_plan(_p(counts), counts.size, n_chunks, max_entries, _p(bounds),
                             bounds.size)
    if nc < 0:
        raise ValueError("chunk plan overflow")
    return bounds[:nc + 1].copy()


def bf16_bits(x: float) -> int:
    return int(lib().or_bf16_bits(C.c_float(x)))
