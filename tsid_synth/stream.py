"""Streaming generators of the observed cells outside the template block.

The Scientific and Billion-scale workloads draw only their template block in
``generate`` (the benchmark times the template fit).  Their extension
(Section 5.2) needs the rest of Omega: every training cell of a free row
against the template columns (row phase) and of a free column against every
row (column phase), 4e9 and about 6e8 cells.  Those are generated here on
demand, a range of free lines at a time, by ``gen.c`` (gcc, OpenMP), so a
phase can be streamed in chunks from host memory without ever holding all of
it:

* Scientific: cell (u, i) is observed when a keyed hash of (u, i) falls below
  0.1, held out when a second keyed hash does, and its value is
  sum_j a_uj s_j b_ij / ||s|| -- the same tests and factors as the template
  block's generator, so template block, row phase and column phase partition
  one Omega.
* Billion-scale: cells of the non-template rows against the template columns
  (row phase) and of every row against the non-template columns (column
  phase) are drawn with the template block's model -- with D pairwise draws
  of Zipf(1.0) popularity, a cell is observed with probability
  1 - exp(-D w_u w_i), independently -- as a Bernoulli prefix plus Poisson
  draws per line, each line from its own counter-based stream; latent
  factors of the non-template rows and columns come from their own seeded
  stream and values are z-scored with the template block's mean and standard
  deviation.

Data only: nothing here computes residuals, gradients or updates.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

from .generate import PURPOSE, Problem, _splitmix64, _zipf_rank_weights, make_rng

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
_LIB = os.path.join(_HERE, "libtsid_gen.so")
_lib: Optional[C.CDLL] = None


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-fopenmp", "-Wall", "-Wextra",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        _lib = C.CDLL(build())
        P, i32, i64, u64, f64 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_double
        _lib.sci_count.restype = None
        _lib.sci_count.argtypes = [i32, P, i64, P, i64, i64, u64, u64, u64, u64, P]
        _lib.sci_fill.restype = None
        _lib.sci_fill.argtypes = [i32, P, i64, P, i64, i32, i64, u64, u64, u64, u64, P, P, i32, P, P, P, P]
        _lib.zipf_cells.restype = C.c_int
        _lib.zipf_cells.argtypes = [P, i64, P, f64, P, P, i64, i64, u64, i32, P, P, i64, u64, u64, i32, P, P, i32,
                                    f64, f64, i32, P, P, P, P, P, i64]
    return _lib


def _p(x):
    return None if x is None else x.ctypes.data_as(C.c_void_p)


def _salt(seed: int, purpose: str) -> int:
    return int(_splitmix64(np.array([seed * 1000003 + PURPOSE[purpose]], dtype=np.uint64))[0])


def _thr(frac: float) -> int:
    return int(frac * (1 << 53))


class Phase:
    """The cells of one extension phase, generated a range of free lines at a
    time.  side 0: free rows against the template columns (fixed id = the
    column's template position); side 1: free columns against every row
    (fixed id = the global row id).  free_ids[f] is the global id of free line
    f; counts[f] its number of training cells."""

    def __init__(self, side, free_ids, counts, fill_fn):
        self.side = side
        self.free_ids = np.ascontiguousarray(free_ids, np.int32)
        self.counts = np.ascontiguousarray(counts, np.int64)
        self.nnz = int(self.counts.sum())
        self._fill = fill_fn

    def fill(self, lo: int, hi: int, fixed: np.ndarray, free_local: np.ndarray, r: np.ndarray) -> int:
        """Writes the cells of free lines [lo, hi), grouped by line, into the
        first entries of the three arrays (free_local relative to lo) and
        returns their number."""
        n = int(self.counts[lo:hi].sum())
        if min(fixed.size, free_local.size, r.size) < n:
            raise ValueError("chunk buffers too small")
        off = np.concatenate([[0], np.cumsum(self.counts[lo:hi])]).astype(np.int64)
        self._fill(lo, hi, off, fixed, free_local, r)
        return n

    def cells(self, lines):
        """(fixed, free_line, r) of the given free lines (indices into
        free_ids), grouped by line in the given order."""
        fixed, fl, rr = [], [], []
        for f in np.asarray(lines, np.int64):
            c = int(self.counts[f])
            a, b, v = np.empty(c, np.int32), np.empty(c, np.int32), np.empty(c, np.float32)
            self.fill(int(f), int(f) + 1, a, b, v)
            fixed.append(a)
            fl.append(np.full(c, f, np.int32))
            rr.append(v)
        return np.concatenate(fixed), np.concatenate(fl), np.concatenate(rr)


class ScientificOmega:
    """The Scientific matrix outside a template block of ``scientific_template``."""

    def __init__(self, p: Problem):
        assert p.name == "scientific"
        self.p = p
        seed = int(p.extra["seed"])
        self.m, self.n, self.k = p.m, p.n, p.k
        gf = make_rng(seed, "factors")
        sig = np.exp(-np.arange(self.k) / 8.0)
        sig = sig / np.linalg.norm(sig)
        self.A = gf.standard_normal((self.m, self.k)).astype(np.float32)
        B = gf.standard_normal((self.n, self.k)).astype(np.float32)
        self.Bs = np.ascontiguousarray(B * sig[None, :].astype(np.float32))
        self.keys = (_salt(seed, "cells"), _thr(0.1), _salt(seed, "holdout"), _thr(0.1))
        row_in = np.zeros(self.m, bool)
        row_in[p.I] = True
        col_in = np.zeros(self.n, bool)
        col_in[p.J] = True
        self.free_rows = np.flatnonzero(~row_in).astype(np.int32)
        self.free_cols = np.flatnonzero(~col_in).astype(np.int32)
        self.J = np.ascontiguousarray(p.J, np.int32)

    def _count(self, is_row, major, minor, n_minor):
        counts = np.empty(major.size, np.int64)
        lib().sci_count(is_row, _p(major), major.size, _p(minor), n_minor, self.n, *self.keys, _p(counts))
        return counts

    def _filler(self, is_row, major, minor, n_minor, ids_out):
        def fill(lo, hi, off, fixed, free_local, r):
            mj = np.ascontiguousarray(major[lo:hi])
            lib().sci_fill(is_row, _p(mj), mj.size, _p(minor), n_minor, ids_out, self.n, *self.keys, _p(self.A),
                           _p(self.Bs), self.k, _p(off), _p(fixed), _p(free_local), _p(r))
        return fill

    def row_phase(self) -> Phase:
        counts = self._count(1, self.free_rows, self.J, self.J.size)
        return Phase(0, self.free_rows, counts, self._filler(1, self.free_rows, self.J, self.J.size, 0))

    def col_phase(self) -> Phase:
        counts = self._count(0, self.free_cols, None, self.m)
        return Phase(1, self.free_cols, counts, self._filler(0, self.free_cols, None, self.m, 1))


class BillionOmega:
    """The Billion-scale matrix outside a template block of ``billion_template``."""

    def __init__(self, p: Problem):
        assert p.name == "billion"
        self.p = p
        seed = int(p.extra["seed"])
        self.m, self.n, self.k = p.m, p.n, p.k
        self.m_t, self.n_t = p.I.size, p.J.size
        self.D = float(p.extra["draws"])
        self.mean, self.sd = float(p.extra["zmean"]), float(p.extra["zstd"])
        self.row_id = make_rng(seed, "rows").permutation(self.m).astype(np.int32)  # id of rank a
        self.col_id = make_rng(seed, "cols").permutation(self.n).astype(np.int32)
        assert np.array_equal(self.row_id[:self.m_t], p.I) and np.array_equal(self.col_id[:self.n_t], p.J)
        self.wr = _zipf_rank_weights(self.m, 1.0)
        self.wc = _zipf_rank_weights(self.n, 1.0)
        self.cwr = np.concatenate([[0.0], np.cumsum(self.wr)])
        self.cwc = np.concatenate([[0.0], np.cumsum(self.wc)])
        # latent factors by rank: the template block's, then the other lines'
        sd = self.k ** -0.25
        gf = make_rng(seed, "factors")
        At = gf.normal(0.0, sd, (self.m_t, self.k)).astype(np.float32)
        Bt = gf.normal(0.0, sd, (self.n_t, self.k)).astype(np.float32)
        ge = make_rng(seed, "extra")
        self.A = np.empty((self.m, self.k), np.float32)
        self.A[:self.m_t] = At
        del At
        for s0 in range(self.m_t, self.m, 1 << 20):  # in slices: the same draws as one call
            s1 = min(self.m, s0 + (1 << 20))
            self.A[s0:s1] = ge.normal(0.0, sd, (s1 - s0, self.k))
        self.B = np.empty((self.n, self.k), np.float32)
        self.B[:self.n_t] = Bt
        self.B[self.n_t:] = ge.normal(0.0, sd, (self.n - self.n_t, self.k))
        self.salt_h, self.thr_h = _salt(seed, "holdout"), _thr(0.1)
        self.key_rows = _salt(seed, "sparse") ^ 0x5257  # streams of the row phase's lines
        self.key_cols = _salt(seed, "sparse") ^ 0x434F  # and of the column phase's

    def _cap(self, wmaj, w, lo, hi):
        lim = np.log(2.0) / (self.D * wmaj)
        pre = int(np.searchsorted(-w[lo:hi], -lim, side="right"))
        lam = self.D * wmaj * (w[lo:hi].sum())
        return int(pre + 4 * lam + 64 * np.sqrt(lam + 1.0) + 4096)

    def _phase(self, side):
        if side == 0:  # free rows (ranks m_t..m) against the template columns (ranks 0..n_t)
            ranks = np.arange(self.m_t, self.m, dtype=np.int64)
            args = (self.wr, self.wc, self.cwc, 0, self.n_t, self.key_rows, 1, self.row_id, self.col_id, 0,
                    self.A, self.B)
            cap = self._cap(self.wr[self.m_t], self.wc, 0, self.n_t)
        else:  # free columns (ranks n_t..n) against every row (ranks 0..m)
            ranks = np.arange(self.n_t, self.n, dtype=np.int64)
            args = (self.wc, self.wr, self.cwr, 0, self.m, self.key_cols, 0, self.col_id, self.row_id, 1,
                    self.B, self.A)
            cap = self._cap(self.wc[self.n_t], self.wr, 0, self.m)
        wmaj, w, cw, lo, hi, key0, is_row, maj_id, min_id, ids_out, Amaj, Bmin = args

        def call(rk, fill, counts, off, fixed, free_local, r):
            st = lib().zipf_cells(_p(rk), rk.size, _p(wmaj), self.D, _p(w), _p(cw), lo, hi, key0, is_row,
                                  _p(maj_id), _p(min_id), self.n, self.salt_h, self.thr_h, ids_out, _p(Amaj),
                                  _p(Bmin), self.k, self.mean, self.sd, fill, _p(counts), _p(off), _p(fixed),
                                  _p(free_local), _p(r), cap)
            if st != 0:
                raise RuntimeError("a line exceeded the generator's capacity")

        counts = np.empty(ranks.size, np.int64)
        call(ranks, 0, counts, None, None, None, None)

        def fill(lo_, hi_, off, fixed, free_local, r):
            call(np.ascontiguousarray(ranks[lo_:hi_]), 1, None, off, fixed, free_local, r)

        return Phase(side, maj_id[ranks], counts, fill)

    def row_phase(self) -> Phase:
        return self._phase(0)

    def col_phase(self) -> Phase:
        return self._phase(1)


def omega_outside_template(p: Problem):
    """The streaming generator of the cells outside p's template block."""
    if p.name == "scientific":
        return ScientificOmega(p)
    if p.name == "billion":
        return BillionOmega(p)
    raise ValueError(f"{p.name}: the whole matrix is drawn by the generator already")
