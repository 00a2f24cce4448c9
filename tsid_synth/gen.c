/*
 * gen.c -- streaming generators of the workloads' observed cells outside the
 * template block (data only: no residuals, gradients, updates or losses).
 *
 * Built by tsid_synth/stream.py with gcc (-O2, OpenMP).  Every routine
 * produces the cells of a list of "major" lines (rows or columns) against a
 * list of "minor" lines, grouped by major line in list order and by minor
 * position within a line, so a caller can generate any range of rows or
 * columns on its own, in any order, and get the same cells.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* SplitMix64's output function (Steele, Lea and Flood, 2014). */
static inline uint64_t mix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* ------------------------------------------------------------ scientific */

/* A cell (u, i) of an n-column matrix is observed when the keyed hash of
 * u * n + i lies below thr_cells (53-bit scale), and held out when the hash
 * with the hold-out key lies below thr_hold; the training cells are the
 * observed ones not held out.  (The Python generator applies the same two
 * tests to the template block.) */
static inline int sci_train(uint64_t u, uint64_t i, uint64_t n, uint64_t salt_c, uint64_t thr_c, uint64_t salt_h,
                            uint64_t thr_h) {
    const uint64_t key = u * n + i;
    if ((mix64(key ^ salt_c) >> 11) >= thr_c) return 0;
    return (mix64(key ^ salt_h) >> 11) >= thr_h;
}

static inline void sci_cell(int major_is_row, int64_t maj, int64_t mi, uint64_t *u, uint64_t *i) {
    if (major_is_row) {
        *u = (uint64_t)maj;
        *i = (uint64_t)mi;
    } else {
        *u = (uint64_t)mi;
        *i = (uint64_t)maj;
    }
}

/* Training cells of each major line against the minor lines (minor NULL:
 * lines 0 .. n_minor - 1). */
void sci_count(int32_t major_is_row, const int32_t *major, int64_t n_major, const int32_t *minor, int64_t n_minor,
               int64_t n, uint64_t salt_c, uint64_t thr_c, uint64_t salt_h, uint64_t thr_h, int64_t *counts) {
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t a = 0; a < n_major; ++a) {
        int64_t c = 0;
        for (int64_t b = 0; b < n_minor; ++b) {
            uint64_t u, i;
            sci_cell(major_is_row, major[a], minor ? minor[b] : b, &u, &i);
            c += sci_train(u, i, (uint64_t)n, salt_c, thr_c, salt_h, thr_h);
        }
        counts[a] = c;
    }
}

/* The cells themselves: cell j of major line a (0-based in the list) goes to
 * offset[a] + j with fixed[] = its minor position b (or minor id when
 * minor_ids_out is set), free_local[] = a, and the value
 * r = sum_c A[u][c] * Bs[i][c] (fp32, c ascending). */
void sci_fill(int32_t major_is_row, const int32_t *major, int64_t n_major, const int32_t *minor, int64_t n_minor,
              int32_t minor_ids_out, int64_t n, uint64_t salt_c, uint64_t thr_c, uint64_t salt_h, uint64_t thr_h,
              const float *A, const float *Bs, int32_t k, const int64_t *offset, int32_t *fixed,
              int32_t *free_local, float *r) {
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t a = 0; a < n_major; ++a) {
        int64_t o = offset[a];
        for (int64_t b = 0; b < n_minor; ++b) {
            const int64_t mi = minor ? minor[b] : b;
            uint64_t u, i;
            sci_cell(major_is_row, major[a], mi, &u, &i);
            if (!sci_train(u, i, (uint64_t)n, salt_c, thr_c, salt_h, thr_h)) continue;
            const float *x = A + u * (uint64_t)k, *y = Bs + i * (uint64_t)k;
            float s = 0.f;
            for (int32_t c = 0; c < k; ++c) s += x[c] * y[c];
            fixed[o] = (int32_t)(minor_ids_out ? mi : b);
            free_local[o] = (int32_t)a;
            r[o] = s;
            ++o;
        }
    }
}

/* --------------------------------------------------------- Zipf pairwise */

/* Counter-based uniform doubles in [0, 1): draw j of stream (key) is
 * mix64(key + j * golden) >> 11, scaled. */
typedef struct {
    uint64_t key, j;
} ustream;

static inline double unif(ustream *s) {
    const uint64_t z = mix64(s->key + (s->j++) * 0x9E3779B97F4A7C15ull);
    return (double)(z >> 11) * (1.0 / 9007199254740992.0);
}

/* Poisson(lam) variates: inversion by sequential search for small means;
 * the transformed rejection method with squeeze (PTRS) of Hormann (1993,
 * "The transformed rejection method for generating Poisson random
 * variables") otherwise. */
static int64_t poisson(ustream *s, double lam) {
    if (lam <= 0.0) return 0;
    if (lam < 10.0) {
        const double e = exp(-lam);
        double p = e, cdf = e, u = unif(s);
        int64_t x = 0;
        while (u > cdf && x < 1000) {
            ++x;
            p *= lam / (double)x;
            cdf += p;
        }
        return x;
    }
    const double slam = sqrt(lam), loglam = log(lam);
    const double b = 0.931 + 2.53 * slam, a = -0.059 + 0.02483 * b;
    const double inv_alpha = 1.1239 + 1.1328 / (b - 3.4), vr = 0.9277 - 3.6224 / (b - 2.0);
    for (;;) {
        const double U = unif(s) - 0.5, V = unif(s);
        const double us = 0.5 - fabs(U);
        const double kx = floor((2.0 * a / us + b) * U + lam + 0.43);
        if (us >= 0.07 && V <= vr) return (int64_t)kx;
        if (kx < 0.0 || (us < 0.013 && V > us)) continue;
        if (log(V) + log(inv_alpha) - log(a / (us * us) + b) <= -lam + kx * loglam - lgamma(kx + 1.0))
            return (int64_t)kx;
    }
}

static int cmp_i64(const void *x, const void *y) {
    const int64_t p = *(const int64_t *)x, q = *(const int64_t *)y;
    return (p > q) - (p < q);
}

/* One major line of rank weight wa against minor ranks [lo, hi) with weights
 * w[] (cumulative cw[r] = w[0] + .. + w[r - 1]): with D pairwise draws a cell
 * is observed with probability 1 - exp(-D wa w_b), independently.  Minor
 * ranks with D wa w_b >= ln 2 (a prefix, weights decreasing) take one
 * Bernoulli trial each; the rest are reached by Poisson(D wa (their total
 * weight)) draws, each picking a rank in proportion to its weight, repeats
 * dropped (each rank then has the same probability).  Writes the observed
 * minor ranks, ascending, to out (capacity cap) and returns their number, or
 * -1 when out is too small. */
static int64_t zipf_line(ustream *s, double D, double wa, const double *w, const double *cw, int64_t lo, int64_t hi,
                         int64_t *out, int64_t cap, int64_t *tmp, int64_t tmp_cap) {
    /* prefix: the first rank (>= lo) with D wa w < ln 2 */
    const double lim = log(2.0) / (D * wa);
    int64_t p0 = lo, p1 = hi;
    while (p0 < p1) {
        const int64_t mid = p0 + (p1 - p0) / 2;
        if (w[mid] >= lim) p0 = mid + 1;
        else p1 = mid;
    }
    const int64_t pre = p0;
    int64_t cnt = 0;
    for (int64_t b = lo; b < pre; ++b)
        if (unif(s) < -expm1(-D * wa * w[b])) {
            if (cnt >= cap) return -1;
            out[cnt++] = b;
        }
    const double rest = cw[hi] - cw[pre];
    const int64_t nd = pre < hi ? poisson(s, D * wa * rest) : 0;
    if (nd > tmp_cap) return -1;
    for (int64_t d = 0; d < nd; ++d) {
        const double y = cw[pre] + unif(s) * rest;
        int64_t q0 = pre, q1 = hi - 1;  /* the rank whose weight interval holds y */
        while (q0 < q1) {
            const int64_t mid = q0 + (q1 - q0) / 2;
            if (cw[mid + 1] <= y) q0 = mid + 1;
            else q1 = mid;
        }
        tmp[d] = q0;
    }
    qsort(tmp, (size_t)nd, sizeof(int64_t), cmp_i64);
    for (int64_t d = 0; d < nd; ++d) {
        if (d > 0 && tmp[d] == tmp[d - 1]) continue;
        if (cnt >= cap) return -1;
        out[cnt++] = tmp[d];
    }
    return cnt;
}

/* Training cells of the major lines of ranks major_rank[0 .. n_major)
 * against the minor ranks [lo, hi), drawn as in zipf_line with the stream of
 * key mix64(key0 ^ rank).  A drawn cell is held out when the keyed hash of
 * its global ids, u * n_cols + i (u, i through the rank permutations), lies
 * below thr_h.  Pass 1 (fill == 0) stores each line's training-cell count;
 * pass 2 (fill == 1) draws the same numbers and writes line a's cells from
 * offset[a] on: fixed = the minor rank (minor_out_ids == 0) or the minor's
 * global id, free_local = a, r = (Amaj[major rank] . Bmin[minor rank] -
 * mean) / sd (fp32 products summed over the coordinates in order).  Returns
 * 0, or -1 when some line had more than line_cap cells or draws. */
int zipf_cells(const int64_t *major_rank, int64_t n_major, const double *wmaj, double D, const double *w,
               const double *cw, int64_t lo, int64_t hi, uint64_t key0, int32_t major_is_row,
               const int32_t *major_id_of_rank, const int32_t *minor_id_of_rank, int64_t n_cols, uint64_t salt_h,
               uint64_t thr_h, int32_t minor_out_ids, const float *Amaj, const float *Bmin, int32_t k, double mean,
               double sd, int32_t fill, int64_t *counts, const int64_t *offset, int32_t *fixed,
               int32_t *free_local, float *r, int64_t line_cap) {
    int bad = 0;
#pragma omp parallel
    {
        int64_t *buf = (int64_t *)malloc((size_t)line_cap * sizeof(int64_t));
        int64_t *tmp = (int64_t *)malloc((size_t)line_cap * sizeof(int64_t));
#pragma omp for schedule(dynamic, 64)
        for (int64_t a = 0; a < n_major; ++a) {
            const int64_t ra = major_rank[a];
            ustream st = {mix64(key0 ^ (uint64_t)ra), 0};
            const int64_t c = zipf_line(&st, D, wmaj[ra], w, cw, lo, hi, buf, line_cap, tmp, line_cap);
            if (c < 0) {
#pragma omp atomic write
                bad = 1;
                continue;
            }
            const uint64_t gmaj = (uint64_t)major_id_of_rank[ra];
            int64_t o = fill ? offset[a] : 0, kept = 0;
            for (int64_t t = 0; t < c; ++t) {
                const int64_t rb = buf[t];
                const uint64_t gmin = (uint64_t)minor_id_of_rank[rb];
                const uint64_t u = major_is_row ? gmaj : gmin, i = major_is_row ? gmin : gmaj;
                if ((mix64((u * (uint64_t)n_cols + i) ^ salt_h) >> 11) < thr_h) continue;  /* held out */
                ++kept;
                if (!fill) continue;
                const float *x = Amaj + ra * (int64_t)k, *y = Bmin + rb * (int64_t)k;
                float sdot = 0.f;
                for (int32_t q = 0; q < k; ++q) sdot += x[q] * y[q];
                fixed[o] = (int32_t)(minor_out_ids ? (int64_t)gmin : rb);
                free_local[o] = (int32_t)a;
                r[o] = (float)(((double)sdot - mean) / sd);
                ++o;
            }
            if (!fill) counts[a] = kept;
        }
        free(buf);
        free(tmp);
    }
    return bad ? -1 : 0;
}
