/*
 * tsid_oracle.h -- plain, serial, fp64 CPU oracle for the TSID template-fit
 * path (arXiv 2608.00977).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library may include,
 * link or call this file; only the tests, the smoke check and the CPU
 * baseline leg of the benchmark use it.  It shares no code with the HIP path.
 *
 * All floating-point arithmetic is IEEE binary64 in straightforward loops.
 * Inputs that arrive as fp32 (values, initial factors) are widened exactly.
 *
 * Status codes match the library's meaning: 0 ok, 1 invalid argument,
 * 2 index out of range, 3 duplicate, 7 non-finite result.
 */
#ifndef TSID_ORACLE_H
#define TSID_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Template index maps (Section 3.1: the index sets I and J; Section 5.1: the
 * sampled column set).  row_map[u] = position of u in I, else -1; likewise
 * col_map.  Range errors take precedence over duplicates. */
int or_template_maps(int64_t m, int64_t n, const int32_t *I, int32_t m_t,
                     const int32_t *J, int32_t n_t, int32_t *row_map, int32_t *col_map);

/* Validates Omega (Definition 1: a set of cells of an m x n matrix):
 * 2 if any (u, i) is out of range, else 1 if any value is not finite,
 * else 3 if a cell repeats, else 0. */
int or_check_omega(int64_t m, int64_t n, int64_t nnz, const int32_t *u, const int32_t *i,
                   const float *r);

/* Omega* = the observed cells inside the template, relabelled to local ids
 * (a, b), in input order (Section 3.2).  Returns |Omega*|. */
int64_t or_filter(int64_t nnz, const int32_t *u, const int32_t *i, const float *r,
                  const int32_t *row_map, const int32_t *col_map,
                  int32_t *a, int32_t *b, float *v);

/* Buckets of Omega* by row (sorted by (a, b)) and by column (sorted by (b, a)),
 * with degrees and exclusive-prefix pointers.  Values are copied bitwise. */
void or_bucket(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
               int32_t m_t, int32_t n_t,
               int64_t *row_ptr, int32_t *csr_col, float *csr_val,
               int64_t *col_ptr, int32_t *csc_row, float *csc_val,
               int32_t *deg_r, int32_t *deg_c);

/* Regularised objective of Section 3.2 (Eq. 2):
 * sum over Omega* of (r - p_a . q_b)^2 + lambda (||P||_F^2 + ||Q||_F^2). */
double or_loss(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
               int32_t m_t, int32_t n_t, int32_t k, const double *P, const double *Q,
               double lambda);

/* Full-gradient (Jacobi) descent on Eq. 2 for `epochs` epochs.
 *   step: 0 = plain gradient step, 1 = per-row/column step scaled by
 *         s = 1/max(1, degree) (the 1/n normalisation of Eq. 5, applied to P
 *         and Q), 2 = the same scale on the columns (Q) only, the rows taking
 *         the plain step, as Eq. 5 prints it.
 *   clip: asymmetric clipping of Section 5.3, min(D, xi) per coordinate of
 *         the descent direction (NaN propagates), D = the row's summed
 *         direction (regulariser once per row, Eq. 2).  1 = after the step
 *         scale: d = min(s D, xi).  3 = before it, the order of the clipped
 *         update as Section 5.3 prints it with eta / n outside the min:
 *         d = s min(D, xi).  2 = per entry, before
 *         the sum (the clipped update of Section 5.3 applied to Eqs. 3-4 entry
 *         by entry): each cell contributes min(2 e q - 2 lambda p, xi) per
 *         coordinate, so the regulariser enters once per cell; the row then
 *         moves by lr s times the sum, and a row without cells stays.
 *   bf16: 1 = the dots and gradient products read bf16 (round-to-nearest-even)
 *         copies of the factors; the fp64 master takes the update.
 * P (m_t x k) and Q (n_t x k) are updated in place; loss_hist (epochs + 1
 * doubles, may be NULL) receives L(P_t, Q_t) for t = 0..epochs.
 * Returns 7 and stops (factors left at the last finite iterate) if an update
 * produces a non-finite value, else 0. */
int or_fit(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
           int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
           int32_t epochs, double lambda, double lr, int32_t step,
           int32_t clip, double xi, int32_t bf16, double *loss_hist, int32_t *epochs_done);

/* or_fit evaluated line by line, for a build with OpenMP: the residuals of
 * all entries, their squares summed in input order, then the gradient sum of
 * every row (and then of every column) over its entries in input order, the
 * lines split across threads, and the row updates.  Each sum has the
 * operands and order of or_fit's, so P, Q and loss_hist are the same bits as
 * or_fit's for any thread count.  Options as or_fit except clip 2 (returns
 * 1) and k > 128 (returns 1). */
int or_fit_lines(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                 int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
                 int32_t epochs, double lambda, double lr, int32_t step,
                 int32_t clip, double xi, int32_t bf16, double *loss_hist, int32_t *epochs_done);

/* Threads an OpenMP build runs its parallel loops with (1 without OpenMP). */
int or_threads(void);

/* Multi-view similarity term (the item-factor update of Section 5.1 with the
 * similarity regulariser of Eq. 1).  S is a symmetric matrix over the
 * template's columns given as COO entries (s_row, s_col, s_val), both
 * orientations listed.  The objective gains
 *   (beta / 2) sum_(i, i') S_ii' ||q_i - q_i'||^2,
 * whose gradient 2 beta sum_i' S_ii' (q_i - q_i') is the printed update term;
 * it joins q_i's summed gradient before the step rule and the clip (modes 0
 * and 1; mode 2 returns 1) and is evaluated at the fp64 master Q.  Ids out
 * of [0, n_t) return 2.  Otherwise as or_fit. */
double or_loss_mv(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                  int32_t m_t, int32_t n_t, int32_t k, const double *P, const double *Q,
                  double lambda, int64_t s_nnz, const int32_t *s_row, const int32_t *s_col,
                  const float *s_val, double beta);
int or_fit_mv(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
              int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
              int32_t epochs, double lambda, double lr, int32_t step,
              int32_t clip, double xi, int32_t bf16, int64_t s_nnz, const int32_t *s_row,
              const int32_t *s_col, const float *s_val, double beta, double *loss_hist,
              int32_t *epochs_done);
/* The item similarity of Section 2.2 from n_attr categorical attributes per
 * item (attr: n x n_attr): S[i][j] = (1 / n_attr) * #{t : attr[i][t] ==
 * attr[j][t]}, dense n x n. */
void or_similarity(int32_t n, int32_t n_attr, const int32_t *attr, double *S);

/* splitmix64 (the published 64-bit finaliser of the SplitMix generator):
 * z = x + 0x9E3779B97F4A7C15, then two xor-shift-multiply rounds and a final
 * xor-shift.  Cell (a, b) of the template (positions in I and J) belongs to
 * mini-batch splitmix64(seed ^ (a << 32 | b)) mod n_batches. */
uint64_t or_splitmix64(uint64_t x);
int32_t or_batch_of(int32_t a, int32_t b, uint64_t seed, int32_t n_batches);
/* or_batch_of for n cells: out[e] = or_batch_of(a[e], b[e], seed, n_batches). */
void or_batch_of_many(int64_t n, const int32_t *a, const int32_t *b, uint64_t seed, int32_t n_batches,
                      int32_t *out);

/* Mini-batch epochs (the in-epoch updates of the stochastic method of
 * Section 5.1, Eq. 5, grouped into mini-batches): each epoch visits the
 * n_batches batches in order and takes, for each, the full-gradient step of
 * or_fit restricted to the batch's cells (the degree step divides by the
 * batch degree, Eq. 5's 1/n over the contributing entries), from the factors
 * the previous batch left; rows and columns without a cell in the batch are
 * not touched.  loss_hist[t] = L(P_t, Q_t) over every cell at the start of
 * epoch t, loss_hist[epochs] at the end.  On a non-finite update the factors
 * are those before the failing batch step, *epochs_done the whole epochs
 * completed, and the status 7. */
int or_fit_minibatch(int64_t nnz, const int32_t *a, const int32_t *b, const float *v,
                     int32_t m_t, int32_t n_t, int32_t k, double *P, double *Q,
                     int32_t epochs, double lambda, double lr, int32_t step,
                     int32_t clip, double xi, int32_t bf16, int32_t n_batches, uint64_t seed,
                     double *loss_hist, int32_t *epochs_done);

/* One-sided extension (Section 5.2, Eq. 6 in factored form): the fixed
 * factors F_fixed (rows indexed by fixed_id) stay constant; each free row
 * f in [0, n_free) starts at zero and takes `steps` gradient steps on
 * sum_{entries of f} (r - F_fixed[id] . x_f)^2 + lambda ||x_f||^2.
 * step 0 or 1 and clip 0, 1 or 3 as for or_fit (the free rows are the side
 * being scaled); step 2 and clip 2 (template-fit options) return 1 untouched. */
int or_extend(int64_t nnz, const int32_t *fixed_id, const int32_t *free_id, const float *v,
              int32_t n_free, int32_t k, const double *F_fixed, double *F_free,
              int32_t steps, double lambda, double lr, int32_t step, int32_t clip, double xi);

/* Exact minimiser of the same per-row ridge problems (normal equations,
 * Cholesky).  Returns 1 if a system is not positive definite. */
int or_ridge(int64_t nnz, const int32_t *fixed_id, const int32_t *free_id, const float *v,
             int32_t n_free, int32_t k, const double *F_fixed, double lambda, double *F_free);

/* Stage II as stated in Section 5.2 (Eq. 6): free line f is represented in
 * the fixed template basis by a coefficient vector c_f (n_b entries), and
 * its entries are predicted as R*_i c_f = p . (B^T c_f), with p the fixed
 * factor row F_fixed[fixed_id] and B (n_b x k) the basis factors of the
 * template (R* = P B^T in factored form).  Minimises
 *   L(C) = sum (r - p . B^T c_f)^2 + lambda ||C||_F^2
 * with the Adam method from C = 0 for `steps` steps: per step the gradient
 * G = dL/dC, the moment estimates m <- beta1 m + (1 - beta1) G and
 * w <- beta2 w + (1 - beta2) G^2, their bias corrections by 1 - beta^t at
 * step t = 1, 2, ..., and C <- C - lr m^ / (sqrt(w^) + eps), elementwise.
 * Outputs F_free[f] = B^T c_f (n_free x k) and, if C_out is not NULL, C
 * (n_free x n_b).  Returns 7 if a coefficient becomes non-finite. */
int or_extend_adam(int64_t nnz, const int32_t *fixed_id, const int32_t *free_id, const float *v,
                   int32_t n_free, int32_t k, const double *F_fixed, int32_t n_b, const double *B,
                   int32_t steps, double lambda, double lr, double beta1, double beta2, double eps,
                   double *F_free, double *C_out);

/* Chunk partition of the free indices (Section 5.2: column chunks processed
 * independently).  counts[f] = entries of free index f, in order.
 * n_chunks > 0: exactly n_chunks runs (some may be empty); run j starts at
 *   the first index f with at least ceil(j * total / n_chunks) entries in
 *   indices before f.
 * else: greedy runs of at most max_entries entries (a single index above the
 *   cap forms its own chunk).
 * bounds receives the start of every chunk plus the end (n_free); returns
 * the number of chunks, or -1 if max_bounds is too small. */
int32_t or_chunk_plan(const int64_t *counts, int64_t n_free, int32_t n_chunks,
                      int64_t max_entries, int64_t *bounds, int32_t max_bounds);

/* bf16 round-to-nearest-even of an fp32 value, returned as the 16-bit pattern. */
uint16_t or_bf16_bits(float x);

#ifdef __cplusplus
}
#endif
#endif
