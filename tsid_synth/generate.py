"""Workload generators (data only; see the package docstring).

Shapes and value models follow the five benchmark configurations:

* ``tiny``        1,000 x 800, rank 8 + N(0, 0.01) noise, 40,000 uniform cells.
* ``mid``         20,000 x 10,000, rank-32 latent model, ratings in {1..5},
                  2.0 M cells with Zipf(1.0) row and column popularity.
* ``rating``      480,189 x 17,770 (the Netflix Prize shape of Section 6.1),
                  100 M cells, Zipf(0.9) rows / Zipf(1.1) columns, rank 64.
* ``scientific``  200,000 x 200,000, rank 32 with singular values exp(-j/8),
                  uniform 10 % observation; only the template block is drawn.
* ``billion``     10 M x 1 M, 1.0e9 cells, Zipf(1.0) rows and columns, rank
                  128, values z-scored; only the 1 M x 100 k template block of
                  the most popular rows and columns is drawn.

Conventions: "N(0, v)" takes v as the variance, so latent factors drawn
N(0, 1/sqrt(k)) give unit-variance products.  Held-out cells are chosen by a
keyed hash of (u, i) so any row range can be regenerated on its own.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, Optional

import numpy as np

PURPOSE = {
    "factors": 1, "rows": 2, "cols": 3, "cells": 4, "values": 5, "noise": 6,
    "holdout": 7, "template": 8, "init": 9, "order": 10, "extra": 11,
    "dense": 12, "sparse": 13,
}


def make_rng(seed: int, purpose: str) -> np.random.Generator:
    """Philox stream keyed by (seed, purpose)."""
    return np.random.Generator(
        np.random.Philox(np.random.SeedSequence([int(seed), PURPOSE[purpose]])))


def _splitmix64(x: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser (Steele, Lea and Flood, 2014) on uint64 arrays."""
    with np.errstate(over="ignore"):
        z = x + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def _cell_hash(u: np.ndarray, i: np.ndarray, n: int, seed: int, purpose: str) -> np.ndarray:
    key = u.astype(np.uint64) * np.uint64(n) + i.astype(np.uint64)
    salt = _splitmix64(np.array([seed * 1000003 + PURPOSE[purpose]], dtype=np.uint64))[0]
    return _splitmix64(key ^ salt)


def _hash_below(h: np.ndarray, frac: float) -> np.ndarray:
    return (h >> np.uint64(11)) < np.uint64(int(frac * (1 << 53)))


def holdout_mask(u: np.ndarray, i: np.ndarray, n: int, seed: int, frac: float = 0.1) -> np.ndarray:
    """True for the ~frac share of cells held out for RMSE (keyed hash of (u, i))."""
    return _hash_below(_cell_hash(u, i, n, seed, "holdout"), frac)


def init_factors(m_t: int, n_t: int, k: int, seed: int):
    """Initial factors P0, Q0 ~ N(0, 1/sqrt(k)) (variance), fp32."""
    g = make_rng(seed, "init")
    sd = k ** -0.25
    P0 = g.normal(0.0, sd, (m_t, k)).astype(np.float32)
    Q0 = g.normal(0.0, sd, (n_t, k)).astype(np.float32)
    return P0, Q0


@dataclasses.dataclass
class Problem:
    """One workload: the training cells of Omega, a held-out split, the
    template index sets (array order = local ids) and the fit settings."""
    name: str
    m: int
    n: int
    u: np.ndarray          # int32, training cells (row ids)
    i: np.ndarray          # int32, training cells (column ids)
    r: np.ndarray          # float32 values
    tu: np.ndarray         # held-out cells
    ti: np.ndarray
    tr: np.ndarray
    I: np.ndarray          # int32 template rows, local order
    J: np.ndarray          # int32 template columns, local order
    k: int
    lam: float
    lr: float
    epochs: int
    step: str              # "sum" | "degree"
    prec: str              # "fp32" | "bf16"
    clip: bool
    xi: float
    P0: np.ndarray         # float32 (len(I), k)
    Q0: np.ndarray         # float32 (len(J), k)
    extra: dict = dataclasses.field(default_factory=dict)

    @property
    def nnz(self) -> int:
        return int(self.u.shape[0])


def _split(u, i, r, n, seed):
    ho = holdout_mask(u, i, n, seed)
    tr = ~ho
    return (u[tr], i[tr], r[tr]), (u[ho], i[ho], r[ho])


def _zipf_cdf(size: int, s: float, g: np.random.Generator) -> np.ndarray:
    """Popularity Zipf(s) by rank, ranks assigned through a seeded permutation."""
    perm = g.permutation(size)
    w = np.empty(size, dtype=np.float64)
    w[perm] = 1.0 / np.power(np.arange(1, size + 1, dtype=np.float64), s)
    c = np.cumsum(w)
    return c / c[-1]


def _inv_cdf(cdf: np.ndarray, x: np.ndarray) -> np.ndarray:
    """First index with cdf > x (numpy's searchsorted 'right'), threaded."""
    import torch
    return torch.searchsorted(torch.from_numpy(cdf), torch.from_numpy(x), right=True).numpy()


def _sorted_distinct(x: np.ndarray) -> np.ndarray:
    """Sorted distinct values of x (what np.unique returns, from one sort)."""
    s = np.sort(x)
    if s.size < 2:
        return s
    keep = np.empty(s.size, dtype=bool)
    keep[0] = True
    np.not_equal(s[1:], s[:-1], out=keep[1:])
    return s[keep]


def _distinct_zipf_cells(m, n, target, cdf_r, cdf_c, g):
    """Exactly `target` distinct cells drawn pairwise from the two
    popularity laws; repeated draws of a cell are discarded and topped up."""
    keys = np.empty(0, dtype=np.int64)
    while keys.size < target:
        need = target - keys.size
        batch = int(need * 2.0) + 65536
        u = _inv_cdf(cdf_r, g.random(batch)).clip(0, m - 1)
        i = _inv_cdf(cdf_c, g.random(batch)).clip(0, n - 1)
        keys = _sorted_distinct(np.concatenate([keys, u.astype(np.int64) * n + i]))
    if keys.size > target:
        keys = np.sort(keys[g.choice(keys.size, target, replace=False)])
    return keys


def _most_observed(ids_deg: np.ndarray, count: int) -> np.ndarray:
    """Indices of the `count` largest degrees, ordered (degree desc, id asc)."""
    ids = np.arange(ids_deg.size)
    order = np.lexsort((ids, -ids_deg.astype(np.int64)))
    return order[:count].astype(np.int32)


def _latent_values(u, i, A, B, chunk=1 << 22):
    """x_e = A[u_e] . B[i_e] for every cell (fp32 products summed by torch's
    multi-threaded CPU kernels; the generator needs speed, not fp64 here)."""
    import torch
    At = torch.from_numpy(np.ascontiguousarray(A, np.float32))
    Bt = torch.from_numpy(np.ascontiguousarray(B, np.float32))
    out = np.empty(u.size, dtype=np.float64)
    n0 = min(chunk, u.size)
    ga = torch.empty((n0, At.shape[1]), dtype=torch.float32)  # reused: no page faults per chunk
    gb = torch.empty((n0, At.shape[1]), dtype=torch.float32)
    dot = torch.empty(n0, dtype=torch.float32)
    for s in range(0, u.size, chunk):
        e = min(u.size, s + chunk)
        n = e - s
        uu = torch.from_numpy(np.ascontiguousarray(u[s:e], np.int64))
        ii = torch.from_numpy(np.ascontiguousarray(i[s:e], np.int64))
        torch.index_select(At, 0, uu, out=ga[:n])
        torch.index_select(Bt, 0, ii, out=gb[:n])
        ga[:n].mul_(gb[:n])
        torch.sum(ga[:n], 1, out=dot[:n])
        out[s:e] = dot[:n].numpy()
    return out


def _finish(name, m, n, u, i, r, seed, I, J, k, settings, extra=None) -> Problem:
    (u_, i_, r_), (tu, ti, tr) = _split(u, i, r, n, seed)
    P0, Q0 = init_factors(I.size, J.size, k, seed)
    return Problem(name=name, m=m, n=n, u=u_.astype(np.int32), i=i_.astype(np.int32),
                   r=r_.astype(np.float32), tu=tu.astype(np.int32), ti=ti.astype(np.int32),
                   tr=tr.astype(np.float32), I=I.astype(np.int32), J=J.astype(np.int32), k=k,
                   P0=P0, Q0=Q0, extra=extra or {}, **settings)


# Fit settings per workload.  Step sizes were fixed once by a sweep of the
# fp64 oracle for a monotone loss (the paper sweeps but does not fix them).
SETTINGS = {
    "tiny": dict(lam=1e-3, lr=0.05, epochs=50, step="sum", prec="fp32", clip=False, xi=0.1),
    "mid": dict(lam=1e-3, lr=0.15, epochs=100, step="degree", prec="fp32", clip=False, xi=0.1),
    "rating": dict(lam=1e-3, lr=0.15, epochs=20, step="degree", prec="bf16", clip=True, xi=0.1),
    "scientific": dict(lam=1e-3, lr=0.5, epochs=20, step="degree", prec="fp32", clip=False, xi=0.1),
    "billion": dict(lam=1e-3, lr=0.1, epochs=20, step="degree", prec="bf16", clip=True, xi=0.1),
}


def tiny(seed: int = 1) -> Problem:
    """1,000 x 800, R = P* Q*^T + N(0, 0.01), 5 % of cells uniform; template
    200 rows x 160 columns drawn uniformly, ascending."""
    m, n, k, nnz = 1000, 800, 8, 40000
    gf = make_rng(seed, "factors")
    sd = k ** -0.25
    A = gf.normal(0.0, sd, (m, k))
    B = gf.normal(0.0, sd, (n, k))
    flat = make_rng(seed, "cells").choice(m * n, nnz, replace=False)
    u, i = flat // n, flat % n
    r = _latent_values(u, i, A, B) + make_rng(seed, "noise").normal(0.0, 0.1, nnz)
    gt = make_rng(seed, "template")
    I = np.sort(gt.choice(m, 200, replace=False))
    J = np.sort(gt.choice(n, 160, replace=False))
    return _finish("tiny", m, n, u, i, r, seed, I, J, k, SETTINGS["tiny"])


def _zipf_rating_problem(name, seed, m, n, nnz, s_row, s_col, rank, m_t, n_t, settings):
    cdf_r = _zipf_cdf(m, s_row, make_rng(seed, "rows"))
    cdf_c = _zipf_cdf(n, s_col, make_rng(seed, "cols"))
    keys = _distinct_zipf_cells(m, n, nnz, cdf_r, cdf_c, make_rng(seed, "cells"))
    keys = keys[make_rng(seed, "order").permutation(keys.size)]
    u = (keys // n).astype(np.int32)
    i = (keys % n).astype(np.int32)
    del keys
    gf = make_rng(seed, "factors")
    sd = rank ** -0.25
    A = gf.normal(0.0, sd, (m, rank)).astype(np.float32)
    B = gf.normal(0.0, sd, (n, rank)).astype(np.float32)
    x = _latent_values(u, i, A, B)
    r = np.rint(np.clip(3.0 + x, 1.0, 5.0))
    del x
    tr_mask = ~holdout_mask(u, i, n, seed)
    I = _most_observed(np.bincount(u[tr_mask], minlength=m), m_t)
    J = _most_observed(np.bincount(i[tr_mask], minlength=n), n_t)
    return _finish(name, m, n, u, i, r, seed, I, J, rank, settings)


def mid(seed: int = 2) -> Problem:
    """20,000 x 10,000, rank-32 latent model, integer ratings 1..5, 2.0 M cells
    with Zipf(1.0) rows and columns; template = top 4,096 x 2,048 by degree."""
    return _zipf_rating_problem("mid", seed, 20000, 10000, 2_000_000, 1.0, 1.0, 32,
                                4096, 2048, SETTINGS["mid"])


def rating(seed: int = 3, scale: float = 1.0) -> Problem:
    """Netflix-Prize-shaped: 480,189 x 17,770, 100 M ratings 1..5, rank 64,
    Zipf(0.9) rows / Zipf(1.1) columns; template 65,536 x 8,192 most observed.
    `scale` < 1 shrinks every size proportionally (test use)."""
    m = max(64, int(480189 * scale))
    n = max(64, int(17770 * scale))
    nnz = max(1000, int(100_000_000 * scale * scale))
    m_t = max(16, int(65536 * scale))
    n_t = max(16, int(8192 * scale))
    return _zipf_rating_problem("rating", seed, m, n, nnz, 0.9, 1.1, 64, m_t, n_t,
                                SETTINGS["rating"])


def scientific_template(seed: int = 4, side: int = 16384, m: int = 200000) -> Problem:
    """200,000 x 200,000 with r_ui = sum_j a_uj s_j b_ij / ||s||, a, b ~ N(0, 1),
    s_j = exp(-j/8), j < 32, each cell observed with probability 0.1 (keyed
    hash).  Only the side x side uniform template block is drawn: membership is
    a per-cell hash, so this block is exactly the template part of the full
    matrix's Omega."""
    n = m
    k = 32
    gt = make_rng(seed, "template")
    I = np.sort(gt.choice(m, side, replace=False)).astype(np.int32)
    J = np.sort(gt.choice(n, side, replace=False)).astype(np.int32)
    gf = make_rng(seed, "factors")
    sig = np.exp(-np.arange(k) / 8.0)
    sig = sig / np.linalg.norm(sig)
    A = gf.standard_normal((m, k)).astype(np.float32)
    B = gf.standard_normal((n, k)).astype(np.float32)
    us, is_, rs = [], [], []
    rows_per = max(1, (1 << 20) // side)
    Ju = J.astype(np.uint64)
    BsT = np.ascontiguousarray((B[J] * sig[None, :].astype(np.float32)).T)
    for a0 in range(0, side, rows_per):
        a1 = min(side, a0 + rows_per)
        uu = I[a0:a1].astype(np.uint64)[:, None]
        keep = _hash_below(_cell_hash(uu, Ju[None, :], n, seed, "cells"), 0.1)
        ra, cb = np.nonzero(keep)
        us.append(I[a0:a1][ra])
        is_.append(J[cb])
        rs.append((A[I[a0:a1]] @ BsT)[ra, cb])
    u = np.concatenate(us)
    i = np.concatenate(is_)
    r = np.concatenate(rs)
    perm = make_rng(seed, "order").permutation(u.size)
    u, i, r = u[perm], i[perm], r[perm]
    return _finish("scientific", m, n, u, i, r, seed, I, J, k, SETTINGS["scientific"],
                   extra={"omega_scope": "template block only", "side": side, "seed": seed})


def _zipf_rank_weights(size: int, s: float) -> np.ndarray:
    """Zipf(s) popularity by rank (rank 1 first), normalised to sum 1."""
    w = 1.0 / np.power(np.arange(1, size + 1, dtype=np.float64), s)
    return w / w.sum()


def _draws_for_distinct(wr: np.ndarray, wc: np.ndarray, target: float, bins: int = 1500) -> float:
    """Number D of independent (row, column) draws, rows ~ wr and columns ~ wc,
    whose expected count of distinct cells is `target`.  A cell drawn with
    probability w_u w_i is seen at least once with probability
    1 - exp(-D w_u w_i); the double sum runs over log-spaced rank bins (each
    bin at its mean weight) and D is found by bisection."""
    def binned(w):
        edges = np.unique(np.round(np.logspace(0, np.log10(w.size), bins)).astype(np.int64) - 1)
        edges = np.append(edges[edges < w.size], w.size)
        cnt = np.diff(edges).astype(np.float64)
        sums = np.add.reduceat(w, edges[:-1])
        return sums / cnt, cnt
    ar, cr = binned(wr)
    ac, cc = binned(wc)
    lo, hi = target, target * 1e4
    for _ in range(80):
        mid = (lo * hi) ** 0.5
        got = np.sum(cr[:, None] * cc[None, :] * -np.expm1(-mid * ar[:, None] * ac[None, :]))
        lo, hi = (mid, hi) if got < target else (lo, mid)
    return (lo * hi) ** 0.5


def _block_rng(seed: int, purpose: str, block: int) -> np.random.Generator:
    """Philox stream keyed by (seed, purpose, block): blocks draw independently,
    so they can be generated in any order or in parallel."""
    return np.random.Generator(
        np.random.Philox(np.random.SeedSequence([int(seed), PURPOSE[purpose], int(block)])))


def billion_template(seed: int = 5, scale: float = 1.0) -> Problem:
    """Billion-scale: 10 M x 1 M, 1.0e9 distinct cells drawn pairwise with
    Zipf(1.0) row and column popularity (ranks through seeded permutations),
    rank 128, values z-scored to N(0, 1).  Template: the 1 M most popular rows
    x the 100 k most popular columns (the expected most-observed ones).

    Only the template block is drawn.  With D pairwise draws (D set so that
    the whole matrix expects 1.0e9 distinct cells) a cell of popularity
    weights w_u, w_i is observed with probability p = 1 - exp(-D w_u w_i),
    independently of the others (the Poisson form of the draws).  Per
    template row, the columns with p >= 1/2 (a prefix, by rank) are kept by a
    Bernoulli trial each; the rest are reached by Poisson(D w_u x their
    weight) draws over those columns, duplicates dropped, which observes each
    with the same p.  Rows are cut into blocks of about 2^24 expected cells,
    each with its own streams; cells come out grouped by row.  `scale` < 1
    shrinks every size (test use)."""
    import torch
    m = max(64, int(10_000_000 * scale))
    n = max(64, int(1_000_000 * scale))
    nnz_full = max(1000.0, 1.0e9 * scale * scale)
    m_t = max(16, int(1_000_000 * scale))
    n_t = max(16, int(100_000 * scale))
    k = 128
    wr = _zipf_rank_weights(m, 1.0)
    wc = _zipf_rank_weights(n, 1.0)
    D = _draws_for_distinct(wr, wc, nnz_full)
    I = make_rng(seed, "rows").permutation(m)[:m_t].astype(np.int32)  # id of rank a
    J = make_rng(seed, "cols").permutation(n)[:n_t].astype(np.int32)
    wr_t, wc_t = wr[:m_t], wc[:n_t]
    C = np.concatenate([[0.0], np.cumsum(wc_t)])   # column weight prefix sums
    Ct = torch.from_numpy(C[1:])
    # dense prefix per row: columns b with D w_a w_b >= ln 2
    K = np.searchsorted(-wc_t, -np.log(2.0) / (D * wr_t), side="right").astype(np.int64)
    lam = D * wr_t * (C[-1] - C[K])                # expected draws past the prefix
    # row blocks of about 2^24 expected cells (dense prefix + sparse draws)
    expect = np.cumsum(K + lam)
    cuts = np.searchsorted(expect, np.arange(1, int(expect[-1] // (1 << 24)) + 1) * float(1 << 24))
    bounds = np.unique(np.concatenate([[0], cuts, [m_t]]))
    parts = []
    for blk in range(bounds.size - 1):
        a0, a1 = int(bounds[blk]), int(bounds[blk + 1])
        gd = _block_rng(seed, "dense", blk)
        gs = _block_rng(seed, "sparse", blk)
        rows = np.arange(a0, a1, dtype=np.int64)
        kd = K[a0:a1]
        rd = np.repeat(rows, kd)
        bd = np.arange(rd.size, dtype=np.int64) - np.repeat(np.cumsum(kd) - kd, kd)
        keep = gd.random(rd.size) < -np.expm1(-D * wr_t[rd] * wc_t[bd])
        dense = rd[keep] * n_t + bd[keep]
        del rd, bd, keep
        rs = np.repeat(rows, gs.poisson(lam[a0:a1]))
        lo = C[K[rs]]
        y = lo + gs.random(rs.size) * (C[-1] - lo)
        bs = torch.searchsorted(Ct, torch.from_numpy(y), right=True).numpy()
        bs = np.clip(bs, K[rs], n_t - 1)
        parts.append(np.sort(np.concatenate([dense, _sorted_distinct(rs * n_t + bs)])))
        del dense, rs, bs, lo, y
    keys = np.concatenate(parts)
    del parts
    a = keys // n_t
    b = keys - a * n_t
    del keys
    gf = make_rng(seed, "factors")
    sd = k ** -0.25
    A = gf.normal(0.0, sd, (m_t, k)).astype(np.float32)
    B = gf.normal(0.0, sd, (n_t, k)).astype(np.float32)
    x = _latent_values(a, b, A, B)
    del A, B
    mu = float(x.mean())
    x -= mu
    sd = float(x.std())
    x /= sd
    u = I[a]
    i = J[b]
    del a, b
    # the cells outside the block (tsid_synth.stream) share D, the z-scoring
    # and the scale
    return _finish("billion", m, n, u, i, x.astype(np.float32), seed, I, J, k, SETTINGS["billion"],
                   extra={"omega_scope": "template block only", "draws": D, "zmean": mu, "zstd": sd,
                          "scale": scale, "seed": seed})


def random_case(m: int, n: int, nnz: int, m_t: int, n_t: int, k: int, seed: int,
                hot_rows: int = 0, hot_cols: int = 0, lam: float = 1e-3, lr: float = 0.2,
                epochs: int = 5, step: str = "degree", prec: str = "fp32", clip: bool = False,
                xi: float = 0.1, holdout: bool = False) -> Problem:
    """Small ragged case for parity tests: `nnz` distinct uniform cells plus
    `hot_rows` fully observed rows and `hot_cols` fully observed columns (so
    buckets far longer than the rest exist); values N(0, 1); the template
    index sets are drawn in random (not ascending) order."""
    g = make_rng(seed, "cells")
    nnz = min(nnz, m * n)
    flat = g.choice(m * n, nnz, replace=False).astype(np.int64)
    extra = []
    if hot_rows:
        for u0 in g.choice(m, hot_rows, replace=False):
            extra.append(u0 * n + np.arange(n, dtype=np.int64))
    if hot_cols:
        for i0 in g.choice(n, hot_cols, replace=False):
            extra.append(np.arange(m, dtype=np.int64) * n + i0)
    if extra:
        flat = np.unique(np.concatenate([flat] + extra))
        flat = flat[make_rng(seed, "order").permutation(flat.size)]
    u, i = flat // n, flat % n
    r = make_rng(seed, "values").standard_normal(flat.size)
    gt = make_rng(seed, "template")
    I = gt.choice(m, m_t, replace=False)
    J = gt.choice(n, n_t, replace=False)
    if hot_rows or hot_cols:
        # put the fully observed rows/columns into the template so its buckets are long
        hr = np.unique(u[np.bincount(u, minlength=m)[u] == n]) if hot_rows else np.empty(0, int)
        hc = np.unique(i[np.bincount(i, minlength=n)[i] == m]) if hot_cols else np.empty(0, int)
        I = np.concatenate([hr, I[~np.isin(I, hr)]])[:m_t]
        J = np.concatenate([hc, J[~np.isin(J, hc)]])[:n_t]
        I = I[make_rng(seed, "extra").permutation(I.size)]
        J = J[make_rng(seed, "extra").permutation(J.size)]
    settings = dict(lam=lam, lr=lr, epochs=epochs, step=step, prec=prec, clip=clip, xi=xi)
    if holdout:
        return _finish("random", m, n, u, i, r, seed, I, J, k, settings)
    P0, Q0 = init_factors(I.size, J.size, k, seed)
    e = np.empty(0, np.int32)
    return Problem(name="random", m=m, n=n, u=u.astype(np.int32), i=i.astype(np.int32),
                   r=r.astype(np.float32), tu=e, ti=e, tr=np.empty(0, np.float32),
                   I=I.astype(np.int32), J=J.astype(np.int32), k=k, P0=P0, Q0=Q0, **settings)


def dense_lowrank_case(m: int, n: int, rank: int, frac: float, seed: int):
    """Noiseless rank-`rank` matrix R = A B^T (A, B ~ N(0, 1/sqrt(rank))) and a
    uniform set of observed cells covering `frac` of R (frac = 1: all).
    Returns (R, u, i)."""
    g = make_rng(seed, "factors")
    sd = rank ** -0.25
    A = g.normal(0.0, sd, (m, rank))
    B = g.normal(0.0, sd, (n, rank))
    R = A @ B.T
    cnt = int(round(frac * m * n))
    flat = np.sort(make_rng(seed, "cells").choice(m * n, cnt, replace=False))
    return R, (flat // n).astype(np.int32), (flat % n).astype(np.int32)


def similarity_graph(n: int, degree: int, seed: int):
    """A random sparse symmetric similarity matrix over n items, as input
    data for the multi-view term: each item links to `degree` others drawn
    uniformly, the links are made mutual, and each pair gets one weight drawn
    uniformly from (0, 1].  Returns COO (row, col, val) with both orientations
    of every pair, no diagonal, no repeated entry."""
    g = make_rng(seed, "extra")
    if n < 2 or degree < 1:
        e = np.empty(0, np.int32)
        return e, e, np.empty(0, np.float32)
    src = np.repeat(np.arange(n, dtype=np.int64), degree)
    dst = (src + g.integers(1, n, src.size)) % n  # never the item itself
    lo, hi = np.minimum(src, dst), np.maximum(src, dst)
    pairs = np.unique(lo * n + hi)
    w = (1.0 - g.random(pairs.size)).astype(np.float32)  # (0, 1]
    a, b = pairs // n, pairs % n
    row = np.concatenate([a, b]).astype(np.int32)
    col = np.concatenate([b, a]).astype(np.int32)
    return row, col, np.concatenate([w, w])


CONFIGS: Dict[str, Callable[..., Problem]] = {
    "tiny": tiny, "mid": mid, "rating": rating, "scientific": scientific_template,
    "billion": billion_template,
}


def make(name: str, seed: Optional[int] = None, **kw) -> Problem:
    fn = CONFIGS[name]
    return fn(**kw) if seed is None else fn(seed=seed, **kw)


_ARRAYS = ("u", "i", "r", "tu", "ti", "tr", "I", "J", "P0", "Q0")


def make_cached(name: str, cache_dir: Optional[str] = None) -> Problem:
    """`make(name)`, kept as plain .npy arrays plus a JSON of the scalar fields
    under cache_dir (None: no cache).  Loading executes nothing from the files
    (numpy without pickles, JSON)."""
    import json
    import os
    if not cache_dir:
        return make(name)
    base = os.path.join(cache_dir, name)
    meta_path = base + ".json"
    if os.path.exists(meta_path):
        meta = json.load(open(meta_path))
        arrs = {a: np.load(f"{base}.{a}.npy", allow_pickle=False) for a in _ARRAYS}
        return Problem(**meta, **arrs)
    p = make(name)
    os.makedirs(cache_dir, exist_ok=True)
    for a in _ARRAYS:
        np.save(f"{base}.{a}.npy", getattr(p, a), allow_pickle=False)
    meta = {f.name: getattr(p, f.name) for f in dataclasses.fields(p) if f.name not in _ARRAYS}
    json.dump(meta, open(meta_path + ".tmp", "w"))
    os.replace(meta_path + ".tmp", meta_path)
    return p
