"""ctypes binding of libtsid (``include/tsid.h``).

Argument marshalling only: every step of the path runs in the HIP library.
The functions named ``tsid_*`` mirror the C entry points one to one; the
:class:`Tsid` class wraps a context for callers holding numpy host arrays
and torch device tensors.  PyTorch is used for device memory, pinned host
memory and streams, nothing else.

The library must be built first (``python -m paper_2608_00977_amd.build``);
loading fails loudly when it is missing -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np
import torch  # imported before libtsid so both share one HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
# TSID_LIB_PATH selects another build of the same library (e.g. a tuning variant).
LIB_PATH = os.environ.get("TSID_LIB_PATH") or os.path.join(_HERE, "libtsid.so")

STATUS = {0: "TSID_OK", 1: "TSID_E_INVAL", 2: "TSID_E_RANGE", 3: "TSID_E_DUP",
          4: "TSID_E_NOMEM", 5: "TSID_E_DEVICE", 6: "TSID_E_STATE", 7: "TSID_E_NONFINITE"}
OK, E_INVAL, E_RANGE, E_DUP, E_NOMEM, E_DEVICE, E_STATE, E_NONFINITE = range(8)
FP32, BF16 = 0, 1
STEP_SUM, STEP_DEGREE, STEP_COL_DEGREE = 0, 1, 2
PASS_KERNEL = {"auto": 0, "item": 1, "slab": 2}
IDX = {"row_map": 0, "col_map": 1, "row_ptr": 2, "csr_col": 3, "csr_val": 4, "col_ptr": 5,
       "csc_row": 6, "csc_val": 7, "deg_r": 8, "deg_c": 9, "batch_ptr_r": 10, "batch_ptr_c": 11}


class TsidError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} {detail}".strip())


class tsid_fit_opts(C.Structure):
    _fields_ = [("epochs", C.c_int32), ("lambda_", C.c_float), ("lr", C.c_float),
                ("clip_xi", C.c_float), ("clip", C.c_int32), ("prec", C.c_int32),
                ("step", C.c_int32)]


class tsid_timing(C.Structure):
    _fields_ = [("pass_ms", C.c_double * 2), ("pass_launches", C.c_int64 * 2),
                ("fixup_ms", C.c_double), ("fixup_launches", C.c_int64),
                ("reduce_ms", C.c_double), ("reduce_launches", C.c_int64),
                ("epoch_ms", C.c_double), ("epochs", C.c_int64),
                ("dense_ms", C.c_double * 2), ("dense_launches", C.c_int64 * 2),
                ("ext_h2d_ms", C.c_double), ("ext_compute_ms", C.c_double), ("ext_chunks", C.c_int64)]


class tsid_adam_opts(C.Structure):
    _fields_ = [("steps", C.c_int32), ("lambda_", C.c_float), ("lr", C.c_float),
                ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float)]


class tsid_dense_info(C.Structure):
    _fields_ = [("cells", C.c_int64), ("tiles", C.c_int64), ("stripes", C.c_int64 * 2)]


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    """Load libtsid.so (built in-tree); raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2608_00977_amd.build` (no fallback exists)")
    L = C.CDLL(LIB_PATH)
    P, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
    sig = {
        "tsid_create": (C.c_int, [C.c_int, P, sz, C.POINTER(P)]),
        "tsid_destroy": (None, [P]),
        "tsid_last_error": (C.c_char_p, [P]),
        "tsid_build_template": (C.c_int, [P, i64, i64, P, P, P, i64, P, i32, P, i32, i32, i64]),
        "tsid_template_info": (C.c_int, [P, P, P, P, P]),
        "tsid_fit_template": (C.c_int, [P, P, P, C.POINTER(tsid_fit_opts), P]),
        "tsid_fit_epochs_done": (C.c_int, [P, P]),
        "tsid_set_timing": (C.c_int, [P, C.c_int]),
        "tsid_set_pass_kernel": (C.c_int, [P, C.c_int]),
        "tsid_fit_pass_kernels": (C.c_int, [P, P, P]),
        "tsid_get_timing": (C.c_int, [P, C.POINTER(tsid_timing)]),
        "tsid_set_dense_tiles": (C.c_int, [P, C.c_float]),
        "tsid_set_minibatch": (C.c_int, [P, i32, C.c_uint64]),
        "tsid_set_similarity": (C.c_int, [P, P, P, P, i64, C.c_float]),
        "tsid_set_row_blocks": (C.c_int, [P, i32]),
        "tsid_fit_row_blocks": (C.c_int, [P, P]),
        "tsid_fit_dense_info": (C.c_int, [P, C.POINTER(tsid_dense_info)]),
        "tsid_loss": (C.c_int, [P, P, P, C.c_float, P]),
        "tsid_loss_noalloc": (C.c_int, [P, P, P, C.c_float, P]),
        "tsid_extend_chunk": (C.c_int, [P, C.c_int, P, P, P, i64, i32, P, i64, P,
                                        C.POINTER(tsid_fit_opts)]),
        "tsid_extend_chunk_ridge": (C.c_int, [P, C.c_int, P, P, P, i64, i32, P, i64, P, C.c_float]),
        "tsid_extend_chunk_adam": (C.c_int, [P, C.c_int, P, P, P, i64, i32, P, i64, P, i64, P, P,
                                             C.POINTER(tsid_adam_opts)]),
        "tsid_sync": (C.c_int, [P]),
        "tsid_export_index": (C.c_int, [P, C.c_int, P, sz]),
        "tsid_chunk_plan": (i32, [P, i64, i32, i64, P, i32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


# ------------------------------------------------------- one-to-one wrappers
def tsid_create(device: int = 0, hip_stream: int = 0, max_device_bytes: int = 0) -> C.c_void_p:
    ctx = C.c_void_p()
    st = lib().tsid_create(device, C.c_void_p(hip_stream or None), max_device_bytes, C.byref(ctx))
    if st != OK:
        raise TsidError(st, "tsid_create")
    return ctx


def tsid_destroy(ctx) -> None:
    lib().tsid_destroy(ctx)


def tsid_last_error(ctx) -> str:
    return lib().tsid_last_error(ctx).decode()


def tsid_build_template(ctx, m, n, u, i, r, nnz, I, m_t, J, n_t, k, stage_entries=0) -> int:
    return lib().tsid_build_template(ctx, m, n, u, i, r, nnz, I, m_t, J, n_t, k, stage_entries)


def tsid_template_info(ctx):
    m_t, n_t, k = C.c_int32(), C.c_int32(), C.c_int32()
    nnz = C.c_int64()
    st = lib().tsid_template_info(ctx, C.byref(m_t), C.byref(n_t), C.byref(nnz), C.byref(k))
    return st, m_t.value, n_t.value, nnz.value, k.value


def tsid_fit_template(ctx, P, Q, opts: tsid_fit_opts, loss_hist) -> int:
    return lib().tsid_fit_template(ctx, P, Q, C.byref(opts), loss_hist)


def tsid_fit_epochs_done(ctx) -> int:
    out = C.c_int32()
    st = lib().tsid_fit_epochs_done(ctx, C.byref(out))
    if st != OK:
        raise TsidError(st, "tsid_fit_epochs_done")
    return out.value


def tsid_set_timing(ctx, every: int) -> int:
    return lib().tsid_set_timing(ctx, int(every))


def tsid_set_pass_kernel(ctx, mode: int) -> int:
    return lib().tsid_set_pass_kernel(ctx, int(mode))


def tsid_fit_pass_kernels(ctx):
    """(P pass, Q pass) kernel names of the last fit ('item', 'slab', or None)."""
    a, b = C.c_int32(0), C.c_int32(0)
    st = lib().tsid_fit_pass_kernels(ctx, C.byref(a), C.byref(b))
    if st != OK:
        raise TsidError(st, "tsid_fit_pass_kernels")
    names = {v: k for k, v in PASS_KERNEL.items()}
    return names.get(a.value), names.get(b.value)


def tsid_get_timing(ctx) -> dict:
    t = tsid_timing()
    st = lib().tsid_get_timing(ctx, C.byref(t))
    if st != OK:
        raise TsidError(st, "tsid_get_timing")
    return dict(pass_ms=[t.pass_ms[0], t.pass_ms[1]],
                pass_launches=[t.pass_launches[0], t.pass_launches[1]],
                fixup_ms=t.fixup_ms, fixup_launches=t.fixup_launches, reduce_ms=t.reduce_ms,
                reduce_launches=t.reduce_launches, epoch_ms=t.epoch_ms, epochs=t.epochs,
                dense_ms=[t.dense_ms[0], t.dense_ms[1]],
                dense_launches=[t.dense_launches[0], t.dense_launches[1]],
                ext_h2d_ms=t.ext_h2d_ms, ext_compute_ms=t.ext_compute_ms, ext_chunks=t.ext_chunks)


def tsid_set_dense_tiles(ctx, fill: float) -> int:
    return lib().tsid_set_dense_tiles(ctx, float(fill))


def tsid_set_minibatch(ctx, n_batches: int, seed: int) -> int:
    return lib().tsid_set_minibatch(ctx, int(n_batches), C.c_uint64(int(seed) & 0xFFFFFFFFFFFFFFFF))


def tsid_set_similarity(ctx, row, col, val, nnz: int, beta: float) -> int:
    return lib().tsid_set_similarity(ctx, row, col, val, int(nnz), float(beta))


def tsid_set_row_blocks(ctx, n_blocks: int) -> int:
    return lib().tsid_set_row_blocks(ctx, int(n_blocks))


def tsid_fit_row_blocks(ctx) -> int:
    out = C.c_int32()
    st = lib().tsid_fit_row_blocks(ctx, C.byref(out))
    if st != OK:
        raise TsidError(st, "tsid_fit_row_blocks")
    return out.value


def tsid_fit_dense_info(ctx) -> dict:
    """Dense tiles of the last fit: cells, tiles, stripes (P pass, Q pass)."""
    d = tsid_dense_info()
    st = lib().tsid_fit_dense_info(ctx, C.byref(d))
    if st != OK:
        raise TsidError(st, "tsid_fit_dense_info")
    return dict(cells=d.cells, tiles=d.tiles, stripes=[d.stripes[0], d.stripes[1]])


def tsid_loss(ctx, P, Q, lam: float, out) -> int:
    return lib().tsid_loss(ctx, P, Q, lam, out)


def tsid_loss_noalloc(ctx, P, Q, lam: float, out) -> int:
    return lib().tsid_loss_noalloc(ctx, P, Q, lam, out)


def tsid_extend_chunk(ctx, side, fixed_id, free_local, r, nnz, n_free, F_fixed, n_fixed, F_free,
                      opts: tsid_fit_opts) -> int:
    return lib().tsid_extend_chunk(ctx, side, fixed_id, free_local, r, nnz, n_free, F_fixed,
                                   n_fixed, F_free, C.byref(opts))


def tsid_extend_chunk_ridge(ctx, side, fixed_id, free_local, r, nnz, n_free, F_fixed, n_fixed,
                            F_free, lam: float) -> int:
    return lib().tsid_extend_chunk_ridge(ctx, side, fixed_id, free_local, r, nnz, n_free, F_fixed,
                                         n_fixed, F_free, float(lam))


def tsid_sync(ctx) -> int:
    return lib().tsid_sync(ctx)


def tsid_export_index(ctx, which: int, host_dst, nbytes: int) -> int:
    return lib().tsid_export_index(ctx, which, host_dst, nbytes)


def tsid_chunk_plan(counts: np.ndarray, n_chunks: int = 0, max_entries: int = 0) -> np.ndarray:
    counts = np.ascontiguousarray(counts, dtype=np.int64)
    cap = (n_chunks + 1) if n_chunks > 0 else counts.size + 2
    bounds = np.empty(max(cap, 2), np.int64)
    nc = lib().tsid_chunk_plan(counts.ctypes.data, counts.size, n_chunks, max_entries,
                               bounds.ctypes.data, bounds.size)
    if nc < 0:
        raise TsidError(E_INVAL, "tsid_chunk_plan")
    return bounds[:nc + 1].copy()


# ------------------------------------------------------------ convenience
def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, torch.Tensor):
        return x.data_ptr()
    return x.ctypes.data


def make_adam_opts(steps=1, lam=0.0, lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8):
    """Options of tsid_extend_chunk_adam (Adam on the coefficients in a basis)."""
    return tsid_adam_opts(int(steps), float(lam), float(lr), float(beta1), float(beta2), float(eps))


CLIP_MODES = {"per_entry": 2, "printed": 3}
STEP_MODES = {"sum": STEP_SUM, "degree": STEP_DEGREE, "col_degree": STEP_COL_DEGREE}


def make_opts(epochs=1, lam=0.0, lr=0.1, clip=False, xi=0.1, prec="fp32", step="sum"):
    """clip: False / True (the clip on each row's normalised summed
    direction), "printed" (the clip on the summed direction before the step
    scale) or "per_entry" (each cell's direction clipped before the sum).
    step: "sum", "degree" or "col_degree"."""
    return tsid_fit_opts(int(epochs), float(lam), float(lr), float(xi),
                         CLIP_MODES[clip] if isinstance(clip, str) else int(bool(clip)),
                         BF16 if prec == "bf16" else FP32,
                         STEP_MODES[step])


class Tsid:
    """One libtsid context on one device."""

    def __init__(self, device: int = 0, stream: Optional[torch.cuda.Stream] = None,
                 max_device_bytes: int = 0):
        torch.cuda.init()
        handle = stream.cuda_stream if stream is not None else 0
        self.device = device
        self.ctx = tsid_create(device, handle, max_device_bytes)
        self._keep = []  # host buffers of chunks in flight

    def close(self):
        if self.ctx is not None:
            tsid_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, st: int, where: str):
        if st != OK:
            raise TsidError(st, where, tsid_last_error(self.ctx))

    def build_template(self, m, n, u, i, r, I, J, k, stage_entries=0):
        u = np.ascontiguousarray(u, np.int32)
        i = np.ascontiguousarray(i, np.int32)
        r = np.ascontiguousarray(r, np.float32)
        I = np.ascontiguousarray(I, np.int32)
        J = np.ascontiguousarray(J, np.int32)
        st = tsid_build_template(self.ctx, m, n, _ptr(u), _ptr(i), _ptr(r), u.size, _ptr(I),
                                 I.size, _ptr(J), J.size, k, stage_entries)
        self._check(st, "tsid_build_template")
        self._dims = (int(m), int(n))

    def info(self):
        st, m_t, n_t, nnz, k = tsid_template_info(self.ctx)
        self._check(st, "tsid_template_info")
        return dict(m_t=m_t, n_t=n_t, nnz=nnz, k=k)

    def fit_template(self, P: torch.Tensor, Q: torch.Tensor, opts: tsid_fit_opts,
                     want_loss: bool = True, raise_on_error: bool = True):
        """Runs the fit in place on P and Q (contiguous fp32 device tensors);
        returns (status, loss history)."""
        assert P.is_cuda and Q.is_cuda and P.dtype == torch.float32 and Q.dtype == torch.float32
        assert P.is_contiguous() and Q.is_contiguous()
        hist = np.full(opts.epochs + 1, np.nan) if want_loss else None
        torch.cuda.current_stream().synchronize()
        st = tsid_fit_template(self.ctx, _ptr(P), _ptr(Q), opts, _ptr(hist))
        if raise_on_error:
            self._check(st, "tsid_fit_template")
        return st, hist

    def set_timing(self, every):
        """Time the kernels of every `every`-th epoch (True: every epoch; 0 /
        False: off); see tsid_set_timing."""
        self._check(tsid_set_timing(self.ctx, int(every)), "tsid_set_timing")

    def set_pass_kernel(self, mode: str):
        """'auto', 'item' or 'slab' (tsid_set_pass_kernel)."""
        self._check(tsid_set_pass_kernel(self.ctx, PASS_KERNEL[mode]), "tsid_set_pass_kernel")

    def pass_kernels(self):
        """Kernels of the last fit's P and Q passes: ('item' | 'slab', ...)."""
        return tsid_fit_pass_kernels(self.ctx)

    def timing(self) -> dict:
        return tsid_get_timing(self.ctx)

    def set_dense_tiles(self, fill: float):
        """Dense head tiles of bf16 fits: fill < 0 automatic, 0 off, in (0, 1]
        forced with that tile fill (tsid_set_dense_tiles)."""
        self._check(tsid_set_dense_tiles(self.ctx, fill), "tsid_set_dense_tiles")

    def set_minibatch(self, n_batches: int, seed: int = 0):
        """Mini-batch epochs: n_batches batches per epoch dealt by a hash of
        each cell's template position and `seed`; 0 restores full-gradient
        epochs (tsid_set_minibatch)."""
        self._check(tsid_set_minibatch(self.ctx, n_batches, seed), "tsid_set_minibatch")
        self._batches = int(n_batches)

    def set_similarity(self, row, col, val, beta: float):
        """Multi-view similarity term: S over the template's columns as COO
        (both orientations listed) and its weight (tsid_set_similarity)."""
        row = np.ascontiguousarray(row, np.int32)
        col = np.ascontiguousarray(col, np.int32)
        val = np.ascontiguousarray(val, np.float32)
        assert row.size == col.size == val.size
        self._check(tsid_set_similarity(self.ctx, _ptr(row), _ptr(col), _ptr(val), val.size, beta),
                    "tsid_set_similarity")

    def set_row_blocks(self, n_blocks: int):
        """Row blocks of the item Q pass: 0 automatic, 1 off, n forced
        (tsid_set_row_blocks)."""
        self._check(tsid_set_row_blocks(self.ctx, n_blocks), "tsid_set_row_blocks")

    def row_blocks(self) -> int:
        """Row blocks the last fit's Q pass ran with (tsid_fit_row_blocks)."""
        return tsid_fit_row_blocks(self.ctx)

    def dense_info(self) -> dict:
        """cells, tiles and stripes (P pass, Q pass) of the last fit's dense
        head tiles (tsid_fit_dense_info)."""
        return tsid_fit_dense_info(self.ctx)

    def epochs_done(self) -> int:
        return tsid_fit_epochs_done(self.ctx)

    def loss(self, P: torch.Tensor, Q: torch.Tensor, lam: float) -> float:
        out = np.zeros(1, np.float64)
        torch.cuda.current_stream().synchronize()
        self._check(tsid_loss(self.ctx, _ptr(P), _ptr(Q), lam, _ptr(out)), "tsid_loss")
        return float(out[0])

    def loss_noalloc(self, P: torch.Tensor, Q: torch.Tensor, lam: float) -> float:
        """tsid_loss_noalloc: the same value from the library's fixed scratch
        array, with no device allocation."""
        out = np.zeros(1, np.float64)
        torch.cuda.current_stream().synchronize()
        self._check(tsid_loss_noalloc(self.ctx, _ptr(P), _ptr(Q), lam, _ptr(out)), "tsid_loss_noalloc")
        return float(out[0])

    def extend_chunk(self, side, fixed_id, free_local, r, n_free, F_fixed: torch.Tensor,
                     F_free: torch.Tensor, opts):
        """Queues one chunk; fixed_id/free_local/r are host arrays or pinned CPU
        tensors kept alive until sync(); F_free receives the result: a CPU
        tensor (pinned for overlap) or a tensor on the context's device.  opts: tsid_fit_opts for the
        one-sided gradient steps (tsid_extend_chunk), or a float lambda for
        the exact ridge solve (tsid_extend_chunk_ridge)."""
        assert F_fixed.is_cuda and F_fixed.dtype == torch.float32 and F_fixed.is_contiguous()
        assert F_free.dtype == torch.float32 and F_free.is_contiguous()
        assert not F_free.is_cuda or F_free.device == F_fixed.device
        arrs = []
        for a, dt in ((fixed_id, np.int32), (free_local, np.int32), (r, np.float32)):
            if isinstance(a, torch.Tensor):
                arrs.append(a)
            else:
                arrs.append(np.ascontiguousarray(a, dt))
        nnz = int(arrs[0].numel() if isinstance(arrs[0], torch.Tensor) else arrs[0].size)
        self._keep.append((arrs, F_fixed, F_free, opts))
        if isinstance(opts, tsid_fit_opts):
            st = tsid_extend_chunk(self.ctx, side, _ptr(arrs[0]), _ptr(arrs[1]), _ptr(arrs[2]), nnz,
                                   n_free, _ptr(F_fixed), F_fixed.shape[0], _ptr(F_free), opts)
            self._check(st, "tsid_extend_chunk")
        else:
            st = tsid_extend_chunk_ridge(self.ctx, side, _ptr(arrs[0]), _ptr(arrs[1]), _ptr(arrs[2]),
                                         nnz, n_free, _ptr(F_fixed), F_fixed.shape[0], _ptr(F_free),
                                         float(opts))
            self._check(st, "tsid_extend_chunk_ridge")

    def extend_chunk_adam(self, side, fixed_id, free_local, r, n_free, F_fixed: torch.Tensor,
                          basis: torch.Tensor, F_free: torch.Tensor, opts: tsid_adam_opts,
                          C_out: Optional[torch.Tensor] = None):
        """Queues one chunk solved by Adam on its coefficients in `basis`
        (tsid_extend_chunk_adam); F_free (and C_out, n_free x n_basis, if given)
        are CPU tensors that receive the results at sync()."""
        assert F_fixed.is_cuda and F_fixed.dtype == torch.float32 and F_fixed.is_contiguous()
        assert basis.is_cuda and basis.dtype == torch.float32 and basis.is_contiguous()
        assert not F_free.is_cuda and F_free.dtype == torch.float32 and F_free.is_contiguous()
        if C_out is not None:
            assert not C_out.is_cuda and C_out.dtype == torch.float32 and C_out.is_contiguous()
        arrs = []
        for a, dt in ((fixed_id, np.int32), (free_local, np.int32), (r, np.float32)):
            arrs.append(a if isinstance(a, torch.Tensor) else np.ascontiguousarray(a, dt))
        nnz = int(arrs[0].numel() if isinstance(arrs[0], torch.Tensor) else arrs[0].size)
        self._keep.append((arrs, F_fixed, basis, F_free, C_out, opts))
        st = lib().tsid_extend_chunk_adam(self.ctx, side, _ptr(arrs[0]), _ptr(arrs[1]), _ptr(arrs[2]), nnz,
                                          n_free, _ptr(F_fixed), F_fixed.shape[0], _ptr(basis),
                                          basis.shape[0], _ptr(F_free),
                                          _ptr(C_out) if C_out is not None else None, C.byref(opts))
        self._check(st, "tsid_extend_chunk_adam")

    def sync(self):
        st = tsid_sync(self.ctx)
        self._keep.clear()
        self._check(st, "tsid_sync")

    def export_index(self, name: str) -> np.ndarray:
        inf = self.info()
        n_rows, n_cols = inf["m_t"], inf["n_t"]
        kind = {"row_map": (np.int32, None), "col_map": (np.int32, None),
                "row_ptr": (np.int64, n_rows + 1), "col_ptr": (np.int64, n_cols + 1),
                "csr_col": (np.int32, inf["nnz"]), "csr_val": (np.float32, inf["nnz"]),
                "csc_row": (np.int32, inf["nnz"]), "csc_val": (np.float32, inf["nnz"]),
                "deg_r": (np.int32, n_rows), "deg_c": (np.int32, n_cols),
                "batch_ptr_r": (np.int64, getattr(self, "_batches", 0) * n_rows + 1),
                "batch_ptr_c": (np.int64, getattr(self, "_batches", 0) * n_cols + 1)}[name]
        count = kind[1] if kind[1] is not None else self._dims[0 if name == "row_map" else 1]
        out = np.empty(count, kind[0])
        self._check(tsid_export_index(self.ctx, IDX[name], _ptr(out), out.nbytes),
                    "tsid_export_index")
        return out
