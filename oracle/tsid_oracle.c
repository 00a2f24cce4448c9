/*
 * tsid_oracle.c -- plain, serial, fp64 CPU oracle for the TSID template-fit
 * path of arXiv 2608.00977 ("TIDE-MC").
 *
 * TEST INFRASTRUCTURE ONLY: called by the tests, the smoke check and the
 * CPU-baseline leg of the benchmark; never by the product library, with which
 * it shares no code.  Every routine is the plain definition or the plain
 * iteration, written as loops, with no blocking, fusion or reordering beyond
 * what the definition states.  Floating point is binary64 throughout.
 *
 * Where the paper leaves a choice open the oracle takes these readings:
 *  - the loss is Eq. 2 literally (regularisation once per factor row);
 *  - the update moves against the gradient of Eqs. 3-4 (descent), applied to
 *    all rows of P and Q simultaneously from the same (P_t, Q_t) (a
 *    deterministic full-gradient epoch);
 *  - the 1/n normalisation of Eq. 5 is the bucket degree, max(1, deg); step
 *    option 1 applies it to both factors, option 2 to the column factors q
 *    only, as Eq. 5 prints it;
 *  - the asymmetric clip of Section 5.3, min(max(xi, -g), g), equals
 *    min(g, xi); option 1 applies it once per coordinate to the aggregated,
 *    normalised descent direction of a row; option 3 applies it to the
 *    aggregated direction before the normalisation, the order in which the
 *    clipped update of Section 5.3 prints the 1/n (outside the min);
 *    option 2 to each entry's own direction before the sum;
 *  - the optional bf16 mode rounds the factors read by the products to bf16
 *    (nearest even) while the fp64 master takes the update.
 */
#include "tsid_oracle.h"

#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- helpers */

typedef struct {
    uint64_t key;
    int64_t idx;
} key_idx;

static int cmp_key_idx(const void *x, const void *y) {
    const key_idx *p = (const key_idx *)x, *q = (const key_idx *)y;
    if (p->key < q->key) return -1;
    if (p->key > q->key) return 1;
    return 0;
}

static int cmp_u64(const void *x, const void *y) {
    uint64_t p = *(const uint64_t *)x, q = *(const uint64_t *)y;
    return (p > q) - (p < q);
}

uint16_t or_bf16_bits(float x) {
    uint32_t bits;
    memcpy(&bits, &x, 4);
    if ((bits & 0x7f800000u) == 0x7f800000u && (bits & 0x007fffffu) != 0)
        return (uint16_t)((bits >> 16) | 0x0040u); /* NaN stays a (quiet) NaN */
    uint32_t lsb = (bits >> 16) & 1u;
    return (uint16_t)((bits + 0x7fffu + lsb) >> 16);
}

static double bf16_round(double x) {
    uint32_t bits = (uint32_t)or_bf16_bits((float)x) << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

static double dot(const double *x, const double *y, int32_t k) {
    double s = 0.0;
    for (int32_t c = 0; c < k; ++c) s += x[c] * y[c];
    return s;
}

static double sumsq(const double *x, int64_t len) {
    double s = 0.0;
    for (int64_t j = 0; j < len; ++j) s += x[j] * x[j];
    return s;
}

/* ------------------------------------------------------------ index work */

int or_template_maps(int64_t m, int64_t n, const int32_t *I, int32_t m_t,
                     const int32_t *J, int32_t n_t, int32_t *row_map, int32_t *col_map) {
    for (int32_t a = 0; a < m_t; ++a)
        if (I[a] < 0 || I[a] >= m) return 2;
    for (int32_t b = 0; b < n_t; ++b)
        if (J[b] < 0 || J[b] >= n) return 2;
    for (int64_t u = 0; u < m; ++u) row_map[u] = -1;
    for (int64_t i = 0; i < n; ++i) col_map[i] = -1;
    for (int32_t a = 0; a < m_t; ++a) {
        if (row_map[I[a]] != -1) return 3;
        row_map[I[a]] = a;
    }
    for (int32_t b = 0; b < n_t; ++b) {
        if (col_map[J[b]] != -1) return 3;
        col_map[J[b]] = b;
    }
    return 0;
}

int or_check_omega(int64_t m, int64_t n, int64_t nnz, const int32_t *u, const int32_t *i,
                   const float *r) {
    for (int64_t e = 0; e < nnz; ++e)
        if (u[e] < 0 || u[e] >= m || i[e] < 0 || i[e] >= n) return 2;
    for (int64_t e = 0; e < nnz; ++e)
        if (!isfinite(r[e])) return 1;
    if (nnz < 2) return 0;
    uint64_t *keys = (uint64_t *)malloc((size_t)nnz * sizeof(uint64_t));
    for (int64_t e = 0; e < nnz; ++e) keys[e] = (uint64_t)u[e] * (uint64_t)n + (uint64_t)i[e];
    qsort(keys, (size_t)nnz, sizeof(uint64_t), cmp_u64);
    int st = 0;
    for (int64_t e = 1; e < nnz; ++e)
        if (keys[e] == keys[e - 1]) { st = 3; break; }
    free(keys);
    return st;
}

int64_t or_filter(int64_t nnz, const int32_t *u, const int32_t *i, const float *r,
                  const int32_t *row_map, const int32_t *col_map,
                  int32_t *a, int32_t *b, float *v) {
    int64_t out = 0;
    for (int64_t e = 0; e < nnz; ++e) {
        int32_t ra = row_map[u[e]], cb = col_map[i[e]];
        if (ra >= 0 && cb >= 0) {
            a[out] = ra;
            b[out] = cb;
            v[out] = r[e];
            ++out;
        }
    }
    return out;
}

/* Sort the entries by (major, minor) and lay them out as buckets of `major`. */
static void bucket_one(int64_t nnz, const int32_t *major, const int32_t *minor, const float *v,
                       int32_t n_major, int32_t n_minor, int64_t *ptr, int32_t *idx_out,
                       float *val_out, int32_t *deg) {
    key_idx *ki = (key_idx *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(key_idx));
    for (int64_t e = 0; e < nnz; ++e) {
        ki[e].key = (uint64_t)major[e] * (uint64_t)n_minor + (uint64_t)minor[e];
        ki[e].idx = e;
    }
    qsort(ki, (size_t)nnz, sizeof(key_idx), cmp_key_idx);
    for (int32_t x = 0; x < n_major; ++x) deg[x] = 0;
    for (int64_t e = 0; e < nnz; ++e) deg[major[e]] += 1;
    ptr[0] = 0;
    for (int32_t x = 0; x < n_major; ++x) ptr[x + 1] = ptr[x] + deg[x];
    for (int64_t e = 0; e < nnz; ++e) {
        idx_out[e] = minor[ki[e].idx];
        val_out[e] = v[ki[e].idx];
    }
    free(ki);
}

void or_bucket(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
               int32_t m_t, int32_t n_t,
               int64_t *row_ptr, int32_t *csr_col, float *csr_val,
               int64_t *col_ptr, int32_t *csc_row, float *csc_val,
               int32_t *deg_r, int32_t *deg_c) {
    bucket_one(nnz, a, b, v, m_t, n_t, row_ptr, csr_col, csr_val, deg_r);
    bucket_one(nnz, b, a, v, n_t, m_t, col_ptr, csc_row, csc_val, deg_c);
}

/* ------------------------------------------------------------------ fit */

double or_loss(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
               int32_t m_t, int32_t n_t, int32_t k, const double *P, const double *Q,
               double lambda) {
    double sse = 0.0;
    for (int64_t e = 0; e < nnz; ++e) {
        double err = (double)v[e] - dot(P + (int64_t)a[e] * k, Q + (int64_t)b[e] * k, k);
        sse += err * err;
    }
    return sse + lambda * (sumsq(P, (int64_t)m_t * k) + sumsq(Q, (int64_t)n_t * k));
}

/* Residual sum of squares over the entries and, if gP/gQ are given, the data
 * part of the gradients of Eqs. 3-4 summed per factor row. */
static double sse_grad(int64_t nnz, const int32_t *a, const int32_t *b, const float *v, int32_t k,
                       const double *Pr, const double *Qr, double *gP, double *gQ) {
    double sse = 0.0;
    for (int64_t e = 0; e < nnz; ++e) {
        const double *p = Pr + (int64_t)a[e] * k, *q = Qr + (int64_t)b[e] * k;
        double err = (double)v[e] - dot(p, q, k);
        sse += err * err;
        if (gP) {
            double *gp = gP + (int64_t)a[e] * k, *gq = gQ + (int64_t)b[e] * k;
            for (int32_t c = 0; c < k; ++c) {
                gp[c] += -2.0 * err * q[c];
                gq[c] += -2.0 * err * p[c];
            }
        }
    }
    return sse;
}

/* Per-entry order of the clipped update (Section 5.3 applied to each entry's
 * own gradient, Eqs. 3-4, before the 1/n average of Eq. 5): cell (p, q) with
 * residual err adds, per coordinate, its descent direction 2 err q - 2 lambda
 * p clipped at xi to the row sums gp, and likewise to gq.  Products use the
 * (possibly bf16-rounded) pr, qr; the regulariser uses the masters p, q. */
static void cell_terms_per_entry(const double *pr, const double *qr, const double *p, const double *q,
                                 double err, int32_t k, double lambda, double xi, double *gp, double *gq) {
    for (int32_t c = 0; c < k; ++c) {
        double dp = 2.0 * err * qr[c] - 2.0 * lambda * p[c];
        double dq = 2.0 * err * pr[c] - 2.0 * lambda * q[c];
        if (dp > xi) dp = xi;
        if (dq > xi) dq = xi;
        gp[c] += dp;
        gq[c] += dq;
    }
}

/* The per-entry sums of every cell (clip mode 2), with the squared residuals. */
static double sse_terms_per_entry(int64_t nnz, const int32_t *a, const int32_t *b, const float *v, int32_t k,
                                  const double *Pr, const double *Qr, const double *P, const double *Q,
                                  double lambda, double xi, double *gP, double *gQ) {
    double sse = 0.0;
    for (int64_t e = 0; e < nnz; ++e) {
        const int64_t oa = (int64_t)a[e] * k, ob = (int64_t)b[e] * k;
        const double err = (double)v[e] - dot(Pr + oa, Qr + ob, k);
        sse += err * err;
        cell_terms_per_entry(Pr + oa, Qr + ob, P + oa, Q + ob, err, k, lambda, xi, gP + oa, gQ + ob);
    }
    return sse;
}

/* Step normalisation s of a factor row with deg observed cells (Eq. 5):
 * step 0 (sum) s = 1; step 1 (degree) s = 1 / max(1, deg) on both sides;
 * step 2 (column degree) the same on the column side (side 1) only. */
static double step_scale(int32_t step, int side, int32_t deg) {
    if (step == 1 || (step == 2 && side == 1)) return 1.0 / (double)(deg > 1 ? deg : 1);
    return 1.0;
}

/* New value of one factor row (Eqs. 3-5, Section 5.3).  clip 0 / 1 / 3: g
 * holds the data gradient -2 sum e q; the regulariser is added once, giving
 * the summed descent direction D = -(g + 2 lambda x); the row moves by lr d
 * with d = s D (clip 0), d = min(s D, xi) (clip 1) or d = s min(D, xi)
 * (clip 3).  clip 2: g holds the clipped per-entry directions, d = s g. */
static int update_row(const double *x, const double *g, int32_t deg, int32_t k, double lambda,
                      double lr, int32_t step, int side, int32_t clip, double xi, double *x_new) {
    const double s = step_scale(step, side, deg);
    int finite = 1;
    for (int32_t c = 0; c < k; ++c) {
        double d;
        if (clip == 2) {
            d = s * g[c];
        } else if (clip == 3) {
            d = -(g[c] + 2.0 * lambda * x[c]);
            if (d > xi) d = xi;
            d = s * d;
        } else {
            d = -s * (g[c] + 2.0 * lambda * x[c]);
            if (clip && d > xi) d = xi;
        }
        x_new[c] = x[c] + lr * d;
        if (!isfinite(x_new[c])) finite = 0;
    }
    return finite;
}

static void round_copy(const double *x, double *y, int64_t len) {
    for (int64_t j = 0; j < len; ++j) y[j] = bf16_round(x[j]);
}

/* ------------------------------------------------ multi-view similarity */

/* The similarity term of the multi-view item update (Section 5.1, with the
 * similarity matrix S of Eq. 1 over the template's columns, symmetric, as COO
 * entries (row[e], col[e], val[e])):
 *   (beta / 2) sum_(i, i') S_ii' ||q_i - q_i'||^2,
 * whose gradient with respect to q_i is 2 beta sum_i' S_ii' (q_i - q_i').
 * Returns the term; adds the gradient to gQ when it is given. */
typedef struct {
    int64_t nnz;
    const int32_t *row, *col;
    const float *val;
    double beta;
} sim_t;

static double sim_terms(const sim_t *S, int32_t k, const double *Q, double *gQ) {
    if (!S) return 0.0;
    double tot = 0.0;
    for (int64_t e = 0; e < S->nnz; ++e) {
        const double *qi = Q + (int64_t)S->row[e] * k, *qj = Q + (int64_t)S->col[e] * k;
        const double w = (double)S->val[e];
        double d2 = 0.0;
        for (int32_t c = 0; c < k; ++c) {
            const double d = qi[c] - qj[c];
            d2 += d * d;
            if (gQ) gQ[(int64_t)S->row[e] * k + c] += 2.0 * S->beta * w * d;
        }
        tot += w * d2;
    }
    return 0.5 * S->beta * tot;
}

void or_similarity(int32_t n, int32_t n_attr, const int32_t *attr, double *S) {
    for (int32_t i = 0; i < n; ++i)
        for (int32_t j = 0; j < n; ++j) {
            int32_t same = 0;
            for (int32_t t = 0; t < n_attr; ++t)
                same += attr[(int64_t)i * n_attr + t] == attr[(int64_t)j * n_attr + t];
            S[(int64_t)i * n + j] = (double)same / (double)n_attr;
        }
}

static int sim_valid(const sim_t *S, int32_t n_t) {
    if (!S) return 1;
    for (int64_t e = 0; e < S->nnz; ++e)
        if (S->row[e] < 0 || S->row[e] >= n_t || S->col[e] < 0 || S->col[e] >= n_t) return 0;
    return 1;
}

double or_loss_mv(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                  int32_t m_t, int32_t n_t, int32_t k, const double *P, const double *Q,
                  double lambda, int64_t s_nnz, const int32_t *s_row, const int32_t *s_col,
                  const float *s_val, double beta) {
    const sim_t S = {s_nnz, s_row, s_col, s_val, beta};
    return or_loss(nnz, a, b, v, m_t, n_t, k, P, Q, lambda) + sim_terms(&S, k, Q, NULL);
}

static int fit_impl(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                    int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
                    int32_t epochs, double lambda, double lr, int32_t step,
                    int32_t clip, double xi, int32_t bf16, const sim_t *S,
                    double *loss_hist, int32_t *epochs_done);

int or_fit(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
           int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
           int32_t epochs, double lambda, double lr, int32_t step,
           int32_t clip, double xi, int32_t bf16, double *loss_hist, int32_t *epochs_done) {
    return fit_impl(nnz, a, b, v, m_t, n_t, k, P, Q, epochs, lambda, lr, step, clip, xi, bf16, NULL,
                    loss_hist, epochs_done);
}

int or_fit_mv(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
              int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
              int32_t epochs, double lambda, double lr, int32_t step,
              int32_t clip, double xi, int32_t bf16, int64_t s_nnz, const int32_t *s_row,
              const int32_t *s_col, const float *s_val, double beta, double *loss_hist,
              int32_t *epochs_done) {
    const sim_t S = {s_nnz, s_row, s_col, s_val, beta};
    if (clip == 2) return 1; /* the per-entry order has no per-entry similarity term */
    if (!sim_valid(&S, n_t)) return 2;
    return fit_impl(nnz, a, b, v, m_t, n_t, k, P, Q, epochs, lambda, lr, step, clip, xi, bf16, &S,
                    loss_hist, epochs_done);
}

static int fit_impl(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                    int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
                    int32_t epochs, double lambda, double lr, int32_t step,
                    int32_t clip, double xi, int32_t bf16, const sim_t *S,
                    double *loss_hist, int32_t *epochs_done) {
    int64_t lp = (int64_t)m_t * k, lq = (int64_t)n_t * k;
    double *gP = (double *)malloc((size_t)(lp + 1) * sizeof(double));
    double *gQ = (double *)malloc((size_t)(lq + 1) * sizeof(double));
    double *Pn = (double *)malloc((size_t)(lp + 1) * sizeof(double));
    double *Qn = (double *)malloc((size_t)(lq + 1) * sizeof(double));
    double *Ps = bf16 ? (double *)malloc((size_t)(lp + 1) * sizeof(double)) : NULL;
    double *Qs = bf16 ? (double *)malloc((size_t)(lq + 1) * sizeof(double)) : NULL;
    int32_t *deg_r = (int32_t *)calloc((size_t)m_t + 1, sizeof(int32_t));
    int32_t *deg_c = (int32_t *)calloc((size_t)n_t + 1, sizeof(int32_t));
    for (int64_t e = 0; e < nnz; ++e) {
        deg_r[a[e]] += 1;
        deg_c[b[e]] += 1;
    }
    int status = 0;
    int32_t t;
    for (t = 0; t < epochs; ++t) {
        const double *Pr = P, *Qr = Q;
        if (bf16) {
            round_copy(P, Ps, lp);
            round_copy(Q, Qs, lq);
            Pr = Ps;
            Qr = Qs;
        }
        memset(gP, 0, (size_t)lp * sizeof(double));
        memset(gQ, 0, (size_t)lq * sizeof(double));
        double sse = clip == 2 ? sse_terms_per_entry(nnz, a, b, v, k, Pr, Qr, P, Q, lambda, xi, gP, gQ)
                               : sse_grad(nnz, a, b, v, k, Pr, Qr, gP, gQ);
        const double sim = sim_terms(S, k, Q, gQ); /* from the fp64 master Q */
        if (loss_hist) loss_hist[t] = sse + lambda * (sumsq(P, lp) + sumsq(Q, lq)) + sim;
        int finite = 1;
        for (int32_t x = 0; x < m_t; ++x)
            finite &= update_row(P + (int64_t)x * k, gP + (int64_t)x * k, deg_r[x], k, lambda, lr,
                                 step, 0, clip, xi, Pn + (int64_t)x * k);
        for (int32_t x = 0; x < n_t; ++x)
            finite &= update_row(Q + (int64_t)x * k, gQ + (int64_t)x * k, deg_c[x], k, lambda, lr,
                                 step, 1, clip, xi, Qn + (int64_t)x * k);
        if (!finite) {
            status = 7;
            break;
        }
        memcpy(P, Pn, (size_t)lp * sizeof(double));
        memcpy(Q, Qn, (size_t)lq * sizeof(double));
    }
    if (status == 0 && loss_hist) {
        const double *Pr = P, *Qr = Q;
        if (bf16) {
            round_copy(P, Ps, lp);
            round_copy(Q, Qs, lq);
            Pr = Ps;
            Qr = Qs;
        }
        double sse = sse_grad(nnz, a, b, v, k, Pr, Qr, NULL, NULL);
        loss_hist[epochs] = sse + lambda * (sumsq(P, lp) + sumsq(Q, lq)) + sim_terms(S, k, Q, NULL);
    }
    if (epochs_done) *epochs_done = t;
    free(gP); free(gQ); free(Pn); free(Qn); free(Ps); free(Qs); free(deg_r); free(deg_c);
    return status;
}

/* ------------------------------------------- line-parallel full-gradient fit */

/* Entry indices of every line (row when major = a, column when major = b),
 * each line's entries in increasing input order (a stable counting sort):
 * ptr[x]..ptr[x+1] index into idx. */
static void lines_in_input_order(int64_t nnz, const int32_t *major, int32_t n_major, int64_t *ptr,
                                 int64_t *idx) {
    for (int32_t x = 0; x <= n_major; ++x) ptr[x] = 0;
    for (int64_t e = 0; e < nnz; ++e) ptr[major[e] + 1] += 1;
    for (int32_t x = 0; x < n_major; ++x) ptr[x + 1] += ptr[x];
    int64_t *fill = (int64_t *)malloc(((size_t)n_major + 1) * sizeof(int64_t));
    memcpy(fill, ptr, ((size_t)n_major + 1) * sizeof(int64_t));
    for (int64_t e = 0; e < nnz; ++e) idx[fill[major[e]]++] = e;
    free(fill);
}

/* or_fit computed line by line: the residual of every entry first, the
 * squared residuals summed in input order, then each row's gradient sum over
 * its entries in input order (rows in parallel when built with OpenMP), the
 * same for columns, and the row updates.  Every sum has the operands and the
 * order of or_fit's, so the results are the same bits; only the work is
 * split across threads.  clip 2 and the similarity term are not offered
 * here (return 1). */
int or_fit_lines(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                 int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
                 int32_t epochs, double lambda, double lr, int32_t step,
                 int32_t clip, double xi, int32_t bf16, double *loss_hist, int32_t *epochs_done) {
    if (clip == 2 || k > 128) return 1;
    const int64_t lp = (int64_t)m_t * k, lq = (int64_t)n_t * k;
    double *Pn = (double *)malloc((size_t)(lp + 1) * sizeof(double));
    double *Qn = (double *)malloc((size_t)(lq + 1) * sizeof(double));
    double *Ps = bf16 ? (double *)malloc((size_t)(lp + 1) * sizeof(double)) : NULL;
    double *Qs = bf16 ? (double *)malloc((size_t)(lq + 1) * sizeof(double)) : NULL;
    double *err = (double *)malloc((size_t)(nnz + 1) * sizeof(double));
    int64_t *rptr = (int64_t *)malloc(((size_t)m_t + 1) * sizeof(int64_t));
    int64_t *cptr = (int64_t *)malloc(((size_t)n_t + 1) * sizeof(int64_t));
    int64_t *ridx = (int64_t *)malloc((size_t)(nnz + 1) * sizeof(int64_t));
    int64_t *cidx = (int64_t *)malloc((size_t)(nnz + 1) * sizeof(int64_t));
    lines_in_input_order(nnz, a, m_t, rptr, ridx);
    lines_in_input_order(nnz, b, n_t, cptr, cidx);
    int status = 0;
    int32_t t;
    for (t = 0; t <= epochs; ++t) {
        const double *Pr = P, *Qr = Q;
        if (bf16) {
#pragma omp parallel for schedule(static)
            for (int64_t j = 0; j < lp; ++j) Ps[j] = bf16_round(P[j]);
#pragma omp parallel for schedule(static)
            for (int64_t j = 0; j < lq; ++j) Qs[j] = bf16_round(Q[j]);
            Pr = Ps;
            Qr = Qs;
        }
#pragma omp parallel for schedule(static)
        for (int64_t e = 0; e < nnz; ++e)
            err[e] = (double)v[e] - dot(Pr + (int64_t)a[e] * k, Qr + (int64_t)b[e] * k, k);
        double sse = 0.0;
        for (int64_t e = 0; e < nnz; ++e) sse += err[e] * err[e];
        if (loss_hist) loss_hist[t] = sse + lambda * (sumsq(P, lp) + sumsq(Q, lq));
        if (t == epochs) break;
        int finite = 1;
#pragma omp parallel for schedule(dynamic, 64) reduction(&& : finite)
        for (int32_t x = 0; x < m_t; ++x) {
            double g[128];
            for (int32_t c = 0; c < k; ++c) g[c] = 0.0;
            for (int64_t j = rptr[x]; j < rptr[x + 1]; ++j) {
                const int64_t e = ridx[j];
                const double *q = Qr + (int64_t)b[e] * k;
                for (int32_t c = 0; c < k; ++c) g[c] += -2.0 * err[e] * q[c];
            }
            finite = update_row(P + (int64_t)x * k, g, (int32_t)(rptr[x + 1] - rptr[x]), k, lambda, lr, step, 0,
                                clip, xi, Pn + (int64_t)x * k) && finite;
        }
#pragma omp parallel for schedule(dynamic, 16) reduction(&& : finite)
        for (int32_t x = 0; x < n_t; ++x) {
            double g[128];
            for (int32_t c = 0; c < k; ++c) g[c] = 0.0;
            for (int64_t j = cptr[x]; j < cptr[x + 1]; ++j) {
                const int64_t e = cidx[j];
                const double *p = Pr + (int64_t)a[e] * k;
                for (int32_t c = 0; c < k; ++c) g[c] += -2.0 * err[e] * p[c];
            }
            finite = update_row(Q + (int64_t)x * k, g, (int32_t)(cptr[x + 1] - cptr[x]), k, lambda, lr, step, 1,
                                clip, xi, Qn + (int64_t)x * k) && finite;
        }
        if (!finite) {
            status = 7;
            break;
        }
        memcpy(P, Pn, (size_t)lp * sizeof(double));
        memcpy(Q, Qn, (size_t)lq * sizeof(double));
    }
    if (epochs_done) *epochs_done = t < epochs ? t : epochs;
    free(Pn); free(Qn); free(Ps); free(Qs); free(err); free(rptr); free(cptr); free(ridx); free(cidx);
    return status;
}

int or_threads(void) {
#ifdef _OPENMP
    int n = 1;
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
    return n;
#else
    return 1;
#endif
}

/* ------------------------------------------------------ mini-batch epochs */

uint64_t or_splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

int32_t or_batch_of(int32_t a, int32_t b, uint64_t seed, int32_t n_batches) {
    const uint64_t key = ((uint64_t)(uint32_t)a << 32) | (uint64_t)(uint32_t)b;
    return (int32_t)(or_splitmix64(seed ^ key) % (uint64_t)n_batches);
}

void or_batch_of_many(int64_t n, const int32_t *a, const int32_t *b, uint64_t seed, int32_t n_batches,
                      int32_t *out) {
    for (int64_t e = 0; e < n; ++e) out[e] = or_batch_of(a[e], b[e], seed, n_batches);
}

int or_fit_minibatch(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                     int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
                     int32_t epochs, double lambda, double lr, int32_t step,
                     int32_t clip, double xi, int32_t bf16, int32_t n_batches, uint64_t seed,
                     double *loss_hist, int32_t *epochs_done) {
    int64_t lp = (int64_t)m_t * k, lq = (int64_t)n_t * k;
    double *gP = (double *)malloc((size_t)(lp + 1) * sizeof(double));
    double *gQ = (double *)malloc((size_t)(lq + 1) * sizeof(double));
    double *Pn = (double *)malloc((size_t)(lp + 1) * sizeof(double));
    double *Qn = (double *)malloc((size_t)(lq + 1) * sizeof(double));
    double *Ps = (double *)malloc((size_t)(lp + 1) * sizeof(double));
    double *Qs = (double *)malloc((size_t)(lq + 1) * sizeof(double));
    int32_t *deg_r = (int32_t *)malloc(((size_t)m_t + 1) * sizeof(int32_t));
    int32_t *deg_c = (int32_t *)malloc(((size_t)n_t + 1) * sizeof(int32_t));
    int32_t *batch = (int32_t *)malloc(((size_t)nnz + 1) * sizeof(int32_t));
    for (int64_t e = 0; e < nnz; ++e) batch[e] = or_batch_of(a[e], b[e], seed, n_batches);
    int status = 0;
    int32_t t;
    for (t = 0; t < epochs && status == 0; ++t) {
        /* L(P_t, Q_t) at the start of the epoch, over every cell */
        const double *Pr = P, *Qr = Q;
        if (bf16) {
            round_copy(P, Ps, lp);
            round_copy(Q, Qs, lq);
            Pr = Ps;
            Qr = Qs;
        }
        if (loss_hist)
            loss_hist[t] = sse_grad(nnz, a, b, v, k, Pr, Qr, NULL, NULL) + lambda * (sumsq(P, lp) + sumsq(Q, lq));
        /* one full-gradient step per batch, on the batch's cells only, each
           from the factors the previous batch left */
        for (int32_t beta = 0; beta < n_batches && status == 0; ++beta) {
            Pr = P;
            Qr = Q;
            if (bf16) {
                round_copy(P, Ps, lp);
                round_copy(Q, Qs, lq);
                Pr = Ps;
                Qr = Qs;
            }
            memset(gP, 0, (size_t)lp * sizeof(double));
            memset(gQ, 0, (size_t)lq * sizeof(double));
            memset(deg_r, 0, ((size_t)m_t + 1) * sizeof(int32_t));
            memset(deg_c, 0, ((size_t)n_t + 1) * sizeof(int32_t));
            for (int64_t e = 0; e < nnz; ++e) {
                if (batch[e] != beta) continue;
                const double *p = Pr + (int64_t)a[e] * k, *q = Qr + (int64_t)b[e] * k;
                const double err = (double)v[e] - dot(p, q, k);
                double *gp = gP + (int64_t)a[e] * k, *gq = gQ + (int64_t)b[e] * k;
                if (clip == 2) {
                    cell_terms_per_entry(p, q, P + (int64_t)a[e] * k, Q + (int64_t)b[e] * k, err, k, lambda, xi,
                                         gp, gq);
                } else {
                    for (int32_t c = 0; c < k; ++c) {
                        gp[c] += -2.0 * err * q[c];
                        gq[c] += -2.0 * err * p[c];
                    }
                }
                deg_r[a[e]] += 1;
                deg_c[b[e]] += 1;
            }
            int finite = 1;
            /* rows and columns without a cell in the batch are not touched */
            for (int32_t x = 0; x < m_t; ++x) {
                if (deg_r[x] == 0) memcpy(Pn + (int64_t)x * k, P + (int64_t)x * k, (size_t)k * sizeof(double));
                else finite &= update_row(P + (int64_t)x * k, gP + (int64_t)x * k, deg_r[x], k, lambda, lr, step,
                                          0, clip, xi, Pn + (int64_t)x * k);
            }
            for (int32_t x = 0; x < n_t; ++x) {
                if (deg_c[x] == 0) memcpy(Qn + (int64_t)x * k, Q + (int64_t)x * k, (size_t)k * sizeof(double));
                else finite &= update_row(Q + (int64_t)x * k, gQ + (int64_t)x * k, deg_c[x], k, lambda, lr, step,
                                          1, clip, xi, Qn + (int64_t)x * k);
            }
            if (!finite) {
                status = 7;
                break;
            }
            memcpy(P, Pn, (size_t)lp * sizeof(double));
            memcpy(Q, Qn, (size_t)lq * sizeof(double));
        }
    }
    if (status) t -= 1; /* the failing epoch did not complete */
    if (status == 0 && loss_hist) {
        const double *Pr = P, *Qr = Q;
        if (bf16) {
            round_copy(P, Ps, lp);
            round_copy(Q, Qs, lq);
            Pr = Ps;
            Qr = Qs;
        }
        loss_hist[epochs] = sse_grad(nnz, a, b, v, k, Pr, Qr, NULL, NULL) + lambda * (sumsq(P, lp) + sumsq(Q, lq));
    }
    if (epochs_done) *epochs_done = t;
    free(gP); free(gQ); free(Pn); free(Qn); free(Ps); free(Qs); free(deg_r); free(deg_c); free(batch);
    return status;
}

/* ------------------------------------------------------------ extension */

int or_extend(int64_t nnz, const int32_t *fixed_id, const int32_t *free_id, const float *v,
              int32_t n_free, int32_t k, const double *F_fixed, double *F_free,
              int32_t steps, double lambda, double lr, int32_t step, int32_t clip, double xi) {
    /* the per-entry clip order and the column-only step are template-fit options */
    if (clip == 2 || step == 2) return 1;
    int64_t len = (int64_t)n_free * k;
    double *g = (double *)malloc((size_t)(len + 1) * sizeof(double));
    double *xn = (double *)malloc((size_t)(len + 1) * sizeof(double));
    int32_t *deg = (int32_t *)calloc((size_t)n_free + 1, sizeof(int32_t));
    for (int64_t e = 0; e < nnz; ++e) deg[free_id[e]] += 1;
    for (int64_t j = 0; j < len; ++j) F_free[j] = 0.0;
    int status = 0;
    for (int32_t s = 0; s < steps && status == 0; ++s) {
        memset(g, 0, (size_t)len * sizeof(double));
        for (int64_t e = 0; e < nnz; ++e) {
            const double *p = F_fixed + (int64_t)fixed_id[e] * k;
            double *x = F_free + (int64_t)free_id[e] * k, *gx = g + (int64_t)free_id[e] * k;
            double err = (double)v[e] - dot(p, x, k);
            for (int32_t c = 0; c < k; ++c) gx[c] += -2.0 * err * p[c];
        }
        int finite = 1;
        for (int32_t f = 0; f < n_free; ++f)
            finite &= update_row(F_free + (int64_t)f * k, g + (int64_t)f * k, deg[f], k, lambda,
                                 lr, step, 0, clip, xi, xn + (int64_t)f * k);
        if (!finite) status = 7;
        else memcpy(F_free, xn, (size_t)len * sizeof(double));
    }
    free(g); free(xn); free(deg);
    return status;
}

int or_ridge(int64_t nnz, const int32_t *fixed_id, const int32_t *free_id, const float *v,
             int32_t n_free, int32_t k, const double *F_fixed, double lambda, double *F_free) {
    int64_t kk = (int64_t)k * k;
    double *A = (double *)calloc((size_t)n_free * kk + 1, sizeof(double));
    double *y = (double *)calloc((size_t)n_free * k + 1, sizeof(double));
    for (int64_t e = 0; e < nnz; ++e) {
        const double *p = F_fixed + (int64_t)fixed_id[e] * k;
        double *Af = A + (int64_t)free_id[e] * kk, *yf = y + (int64_t)free_id[e] * k;
        for (int32_t r = 0; r < k; ++r) {
            yf[r] += (double)v[e] * p[r];
            for (int32_t c = 0; c < k; ++c) Af[r * k + c] += p[r] * p[c];
        }
    }
    int status = 0;
    for (int32_t f = 0; f < n_free && status == 0; ++f) {
        double *M = A + (int64_t)f * kk, *rhs = y + (int64_t)f * k, *x = F_free + (int64_t)f * k;
        for (int32_t r = 0; r < k; ++r) M[r * k + r] += lambda;
        /* Cholesky M = L L^T, L stored in the lower triangle of M. */
        for (int32_t j = 0; j < k && status == 0; ++j) {
            double d = M[j * k + j];
            for (int32_t c = 0; c < j; ++c) d -= M[j * k + c] * M[j * k + c];
            if (!(d > 0.0)) { status = 1; break; }
            double ljj = sqrt(d);
            M[j * k + j] = ljj;
            for (int32_t r = j + 1; r < k; ++r) {
                double s = M[r * k + j];
                for (int32_t c = 0; c < j; ++c) s -= M[r * k + c] * M[j * k + c];
                M[r * k + j] = s / ljj;
            }
        }
        if (status) break;
        for (int32_t r = 0; r < k; ++r) { /* L z = rhs */
            double s = rhs[r];
            for (int32_t c = 0; c < r; ++c) s -= M[r * k + c] * x[c];
            x[r] = s / M[r * k + r];
        }
        for (int32_t r = k - 1; r >= 0; --r) { /* L^T x = z */
            double s = x[r];
            for (int32_t c = r + 1; c < k; ++c) s -= M[c * k + r] * x[c];
            x[r] = s / M[r * k + r];
        }
    }
    free(A); free(y);
    return status;
}

int or_extend_adam(int64_t nnz, const int32_t *fixed_id, const int32_t *free_id, const float *v,
                   int32_t n_free, int32_t k, const double *F_fixed, int32_t n_b, const double *B,
                   int32_t steps, double lambda, double lr, double beta1, double beta2, double eps,
                   double *F_free, double *C_out) {
    const int64_t nc = (int64_t)n_free * n_b, nx = (int64_t)n_free * k;
    double *C = (double *)calloc((size_t)nc + 1, sizeof(double));
    double *m = (double *)calloc((size_t)nc + 1, sizeof(double));
    double *w = (double *)calloc((size_t)nc + 1, sizeof(double));
    double *gt = (double *)malloc((size_t)(nx + 1) * sizeof(double));
    int status = 0;
    double b1t = 1.0, b2t = 1.0;
    for (int32_t t = 1; t <= steps && status == 0; ++t) {
        /* x_f = B^T c_f, the factor the coefficients represent */
        for (int32_t f = 0; f < n_free; ++f)
            for (int32_t c = 0; c < k; ++c) {
                double s = 0.0;
                for (int32_t l = 0; l < n_b; ++l) s += B[(int64_t)l * k + c] * C[(int64_t)f * n_b + l];
                F_free[(int64_t)f * k + c] = s;
            }
        /* dL/dx_f = -2 sum (r - p . x_f) p over the entries of f */
        memset(gt, 0, (size_t)nx * sizeof(double));
        for (int64_t e = 0; e < nnz; ++e) {
            const double *p = F_fixed + (int64_t)fixed_id[e] * k;
            const int64_t f = free_id[e];
            const double err = (double)v[e] - dot(p, F_free + f * k, k);
            for (int32_t c = 0; c < k; ++c) gt[f * k + c] += -2.0 * err * p[c];
        }
        /* dL/dc_f = B dL/dx_f + 2 lambda c_f, then the Adam step */
        b1t *= beta1;
        b2t *= beta2;
        for (int32_t f = 0; f < n_free; ++f)
            for (int32_t l = 0; l < n_b; ++l) {
                const int64_t j = (int64_t)f * n_b + l;
                const double g = dot(B + (int64_t)l * k, gt + (int64_t)f * k, k) + 2.0 * lambda * C[j];
                m[j] = beta1 * m[j] + (1.0 - beta1) * g;
                w[j] = beta2 * w[j] + (1.0 - beta2) * g * g;
                const double mh = m[j] / (1.0 - b1t), wh = w[j] / (1.0 - b2t);
                C[j] -= lr * mh / (sqrt(wh) + eps);
                if (!isfinite(C[j])) status = 7;
            }
    }
    for (int32_t f = 0; f < n_free; ++f)
        for (int32_t c = 0; c < k; ++c) {
            double s = 0.0;
            for (int32_t l = 0; l < n_b; ++l) s += B[(int64_t)l * k + c] * C[(int64_t)f * n_b + l];
            F_free[(int64_t)f * k + c] = s;
        }
    if (C_out) memcpy(C_out, C, (size_t)nc * sizeof(double));
    free(C); free(m); free(w); free(gt);
    return status;
}

int32_t or_chunk_plan(const int64_t *counts, int64_t n_free, int32_t n_chunks,
                      int64_t max_entries, int64_t *bounds, int32_t max_bounds) {
    if (n_chunks > 0) {
        if (max_bounds < n_chunks + 1) return -1;
        int64_t total = 0;
        for (int64_t f = 0; f < n_free; ++f) total += counts[f];
        int64_t before = 0, f = 0;
        bounds[0] = 0;
        for (int32_t j = 1; j < n_chunks; ++j) {
            /* ceil(j * total / n_chunks) without overflow for realistic sizes */
            int64_t target = (int64_t)(((__int128)j * total + n_chunks - 1) / n_chunks);
            while (f < n_free && before < target) before += counts[f++];
            bounds[j] = f;
        }
        bounds[n_chunks] = n_free;
        return n_chunks;
    }
    int32_t nb = 0;
    if (max_bounds < 1) return -1;
    bounds[nb++] = 0;
    if (n_free == 0) return 0;
    int64_t in_chunk = 0, rows_in_chunk = 0;
    for (int64_t f = 0; f < n_free; ++f) {
        if (rows_in_chunk > 0 && in_chunk + counts[f] > max_entries) {
            if (nb >= max_bounds) return -1;
            bounds[nb++] = f;
            in_chunk = 0;
            rows_in_chunk = 0;
        }
        in_chunk += counts[f];
        rows_in_chunk += 1;
    }
    if (nb >= max_bounds) return -1;
    bounds[nb++] = n_free;
    return nb - 1;
}
