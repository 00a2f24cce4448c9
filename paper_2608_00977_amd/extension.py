"""End-to-end extension of the template factors to the whole matrix
(Section 5.2), on top of ``tsid_extend_chunk`` and ``tsid_chunk_plan``.

Order of the two phases (every training cell outside the template block is
used exactly once):

* row phase: each row not in the template is fitted from its cells in
  template columns, with the template column factors Q_J fixed;
* column phase: each column not in the template is fitted from all of its
  cells, with every row factor fixed (template rows from the fit, the other
  rows from the row phase).

Each phase groups its cells by free index on the host, cuts them into
chunks of whole rows (or columns) with ``tsid_chunk_plan`` and streams the
chunks through the library, which stages each chunk's host-to-device copy on
its own stream while the previous chunk computes.  This module only slices
and pins host arrays; all arithmetic runs in the library's kernels.
"""
import time
from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np
import torch

from .binding import Tsid, tsid_adam_opts, tsid_chunk_plan


@dataclass
class Phase:
    side: int                 # 0: free rows (fixed: template columns); 1: free columns
    free_ids: np.ndarray      # global ids of the free rows / columns, ascending
    bounds: np.ndarray        # chunk boundaries in free-index space
    nnz: int
    chunks: List[Tuple[torch.Tensor, torch.Tensor, torch.Tensor, int, int]] = field(
        default_factory=list)  # (fixed_id, free_local, r) pinned, free range [lo, hi)


def _phase(side, free_mask, key, fixed, r, n_chunks, max_entries) -> Phase:
    free_ids = np.flatnonzero(free_mask)
    pos = np.full(free_mask.size, -1, np.int64)
    pos[free_ids] = np.arange(free_ids.size)
    fk = pos[key]
    # each free line's cells together, fixed ids ascending within a line: the
    # library then finds every chunk already in its bucket order and skips
    # the device sort.  One sort of a combined (line, fixed id) key (repeated
    # cells, an error the library reports, stay neighbours in any order).
    nbits = max(1, int(fixed.max()).bit_length()) if fixed.size else 1
    order = np.argsort((fk << nbits) | fixed.astype(np.int64), kind="quicksort")
    fk, fixed, r = fk[order], fixed[order], r[order]
    counts = np.bincount(fk, minlength=free_ids.size).astype(np.int64)
    bounds = tsid_chunk_plan(counts, n_chunks, max_entries)
    start = np.concatenate([[0], np.cumsum(counts)])
    ph = Phase(side, free_ids, bounds, int(fk.size))
    for j in range(bounds.size - 1):
        lo, hi = int(bounds[j]), int(bounds[j + 1])
        e0, e1 = int(start[lo]), int(start[hi])
        pin = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dt)).pin_memory()
        ph.chunks.append((pin(fixed[e0:e1], np.int32), pin(fk[e0:e1] - lo, np.int32),
                          pin(r[e0:e1], np.float32), lo, hi))
    return ph


class Extension:
    """Host plan of both phases for one matrix and template (built once;
    ``run`` may be called repeatedly, e.g. with new template factors)."""

    def __init__(self, m, n, u, i, r, I, J, n_chunks=16, max_entries=0):
        u = np.asarray(u, np.int64)
        i = np.asarray(i, np.int64)
        r = np.asarray(r, np.float32)
        self.m, self.n = int(m), int(n)
        self.I = np.asarray(I, np.int64)
        self.J = np.asarray(J, np.int64)
        row_in = np.zeros(self.m, bool)
        row_in[self.I] = True
        col_in = np.zeros(self.n, bool)
        col_in[self.J] = True
        cm = np.full(self.n, -1, np.int64)
        cm[self.J] = np.arange(self.J.size)
        sel = ~row_in[u] & col_in[i]
        self.rows = _phase(0, ~row_in, u[sel], cm[i[sel]], r[sel], n_chunks, max_entries)
        sel = ~col_in[i]
        self.cols = _phase(1, ~col_in, i[sel], u[sel], r[sel], n_chunks, max_entries)
        self.template_nnz = int(np.count_nonzero(row_in[u] & col_in[i]))

    def _run_phase(self, T: Tsid, ph: Phase, F_fixed: torch.Tensor, out: torch.Tensor, opts,
                   basis: torch.Tensor):
        for fx, fl, rr, lo, hi in ph.chunks:
            if isinstance(opts, tsid_adam_opts):
                T.extend_chunk_adam(ph.side, fx, fl, rr, hi - lo, F_fixed, basis, out[lo:hi], opts)
            else:
                T.extend_chunk(ph.side, fx, fl, rr, hi - lo, F_fixed, out[lo:hi], opts)
        T.sync()

    def run(self, T: Tsid, P_t: torch.Tensor, Q_t: torch.Tensor, opts, col_opts=None):
        """P_t (m_t x k), Q_t (n_t x k): fp32 device factors of the template,
        in template order.  opts (and col_opts for the column phase, if given):
        tsid_fit_opts for one-sided gradient steps, a float lambda for the
        exact ridge solve of every free line, or tsid_adam_opts for Adam on
        the coefficients of each free line in the template basis (Eq. 6:
        free columns over the template columns' factors Q_t, free rows over
        the template rows' factors P_t).  Returns (P, Q): the full m x k and n x k factors
        as pinned host tensors, and the wall time of each phase in seconds.
        The row phase's factors stay on the device for the column phase
        (steps and the exact solve; the Adam path returns them to the host)."""
        k = P_t.shape[1]
        adam = isinstance(opts, tsid_adam_opts)
        P_free = (torch.empty((self.rows.free_ids.size, k), dtype=torch.float32).pin_memory() if adam
                  else torch.empty((self.rows.free_ids.size, k), dtype=torch.float32, device=P_t.device))
        Q_free = torch.empty((self.cols.free_ids.size, k), dtype=torch.float32).pin_memory()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        self._run_phase(T, self.rows, Q_t, P_free, opts, P_t)
        t1 = time.perf_counter()
        P_full = torch.empty((self.m, k), dtype=torch.float32, device=P_t.device)
        P_full[torch.from_numpy(self.I).to(P_t.device)] = P_t
        if self.rows.free_ids.size:
            P_full[torch.from_numpy(self.rows.free_ids).to(P_t.device)] = P_free.to(P_t.device, non_blocking=True)
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        self._run_phase(T, self.cols, P_full, Q_free, opts if col_opts is None else col_opts, Q_t)
        t3 = time.perf_counter()
        P = P_full.cpu()
        Q = torch.empty((self.n, k), dtype=torch.float32)
        Q[torch.from_numpy(self.J)] = Q_t.cpu()
        if self.cols.free_ids.size:
            Q[torch.from_numpy(self.cols.free_ids)] = Q_free
        return P, Q, {"row_phase_s": t1 - t0, "assemble_s": t2 - t1, "col_phase_s": t3 - t2}


def _pinned(n, dtype):
    return torch.empty(max(1, int(n)), dtype=dtype).pin_memory()


class StreamedExtension:
    """Both phases of the extension from sources that produce their cells a
    range of free lines at a time, for matrices whose Omega is not held in
    memory (Section 5.2: the matrix is processed in chunks streamed from the
    host).  A source is any object with ``side`` (0 rows, 1 columns),
    ``free_ids`` (global id of each free line), ``counts`` (cells per free
    line) and ``fill(lo, hi, fixed, free_local, r)`` writing the cells of free
    lines [lo, hi) -- fixed ids as the phase's F_fixed expects them -- and
    returning their number.

    Chunks are runs of whole free lines of at most ``max_entries`` cells
    (``tsid_chunk_plan``).  By default each chunk is filled into one of two
    pinned host buffers just before it is queued; ``tsid_extend_chunk``
    returns once the previous chunk's copy has finished, so the other buffer
    is then free for the next chunk while this one copies and the previous
    one computes.  With ``prefill`` every chunk is filled into pinned memory
    up front (``prefill_s``), and ``run`` times the stream alone."""

    def __init__(self, m, n, I, J, rows, cols, max_entries, prefill=False):
        self.m, self.n = int(m), int(n)
        self.I = np.asarray(I, np.int64)
        self.J = np.asarray(J, np.int64)
        self.rows, self.cols = rows, cols
        self.bounds = [tsid_chunk_plan(np.asarray(ph.counts, np.int64), 0, int(max_entries)) for ph in (rows, cols)]
        self.prefill_s = 0.0
        self.chunks = None
        self.fill_s = [0.0, 0.0]
        if prefill:
            t0 = time.perf_counter()
            self.chunks = [self._fill_all(ph, b) for ph, b in zip((rows, cols), self.bounds)]
            self.prefill_s = time.perf_counter() - t0
        else:
            cap = max(self._largest(ph, b) for ph, b in zip((rows, cols), self.bounds))
            self.buf = [(_pinned(cap, torch.int32), _pinned(cap, torch.int32), _pinned(cap, torch.float32))
                        for _ in range(2)]

    @staticmethod
    def _largest(ph, bounds):
        c = np.concatenate([[0], np.cumsum(np.asarray(ph.counts, np.int64))])
        return int(max((c[bounds[j + 1]] - c[bounds[j]] for j in range(bounds.size - 1)), default=0))

    @staticmethod
    def _fill_all(ph, bounds):
        fx, fl, rr = _pinned(ph.nnz, torch.int32), _pinned(ph.nnz, torch.int32), _pinned(ph.nnz, torch.float32)
        out, e0 = [], 0
        for j in range(bounds.size - 1):
            lo, hi = int(bounds[j]), int(bounds[j + 1])
            n = ph.fill(lo, hi, fx[e0:].numpy(), fl[e0:].numpy(), rr[e0:].numpy())
            out.append((fx[e0:e0 + n], fl[e0:e0 + n], rr[e0:e0 + n], lo, hi))
            e0 += n
        return out

    def _run_phase(self, T: Tsid, which, F_fixed, out, opts):
        ph, bounds = (self.rows, self.cols)[which], self.bounds[which]
        for j in range(bounds.size - 1):
            lo, hi = int(bounds[j]), int(bounds[j + 1])
            if self.chunks is not None:
                fx, fl, rr, _, _ = self.chunks[which][j]
            else:
                b = self.buf[j % 2]
                t0 = time.perf_counter()
                n = ph.fill(lo, hi, b[0].numpy(), b[1].numpy(), b[2].numpy())
                self.fill_s[which] += time.perf_counter() - t0
                fx, fl, rr = b[0][:n], b[1][:n], b[2][:n]
            if isinstance(opts, tsid_adam_opts):
                raise ValueError("the streamed extension runs the factored solvers")
            T.extend_chunk(ph.side, fx, fl, rr, hi - lo, F_fixed, out[lo:hi], opts)
        T.sync()

    def run(self, T: Tsid, P_t: torch.Tensor, Q_t: torch.Tensor, opts, col_opts=None):
        """P_t (m_t x k), Q_t (n_t x k): fp32 device factors of the template.
        opts (and col_opts for the column phase): tsid_fit_opts for one-sided
        gradient steps, or a float lambda for the exact ridge solve.  Returns
        P_full (m x k, device: the template rows and the row phase's), P_free
        and Q_free (the two phases' free lines, on the device and in pinned host
        memory, in the sources'
        order) and the wall time of each phase in seconds (with the time spent
        filling host buffers, when not prefilled).  P_free stays on the device
        (the column phase reads it there): 9 M x 128 fp32 rows are 4.6 GB of
        HBM instead of a return trip over PCIe."""
        k = P_t.shape[1]
        P_free = torch.empty((self.rows.free_ids.size, k), dtype=torch.float32, device=P_t.device)
        Q_free = _pinned(self.cols.free_ids.size * k, torch.float32)[:self.cols.free_ids.size * k].view(-1, k)
        self.fill_s = [0.0, 0.0]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        self._run_phase(T, 0, Q_t, P_free, opts)
        t1 = time.perf_counter()
        P_full = torch.empty((self.m, k), dtype=torch.float32, device=P_t.device)
        P_full[torch.from_numpy(self.I).to(P_t.device)] = P_t
        if self.rows.free_ids.size:
            P_full[torch.from_numpy(np.asarray(self.rows.free_ids, np.int64)).to(P_t.device)] = P_free
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        self._run_phase(T, 1, P_full, Q_free, opts if col_opts is None else col_opts)
        t3 = time.perf_counter()
        return P_full, P_free, Q_free, {"row_phase_s": t1 - t0, "assemble_s": t2 - t1, "col_phase_s": t3 - t2,
                                        "row_fill_s": self.fill_s[0], "col_fill_s": self.fill_s[1]}
