/*
 * tsid.h -- C ABI of libtsid, the MI355X (gfx950) implementation of the
 * data-parallel hot path of TSID matrix completion (arXiv 2608.00977,
 * "TIDE-MC"): the template fit of Stage I and the chunked one-sided extension
 * of Stage II.
 *
 * Problem statement (Definition 1, Section 2): R is m x n; the observed cells
 * Omega are given as COO triples (u, i, r) with 0 <= u < m, 0 <= i < n, each
 * cell at most once.  A template is fixed by index sets I (rows) and J
 * (columns) (Section 3.1); Omega* is the part of Omega inside I x J
 * (Section 3.2).  Local ids follow the array order of I and J: row I[a] of R is
 * template row a.
 *
 * Conventions for every call:
 *  - Every call returns a tsid_status; TSID_OK == 0.  Calls on one context are
 *    not thread-safe; separate contexts are independent.
 *  - The caller owns every pointer it passes.  The context owns all device
 *    memory it allocates (maps, buckets, staging, factor copies, scratch) and
 *    frees it in tsid_destroy.
 *  - "HOST" pointers are CPU memory (pinned memory is faster for the bulk
 *    arrays); "DEVICE" pointers are device memory on the context's device.
 *  - Factor matrices are row-major fp32 with k columns.
 *  - Arguments are validated before any device work.  On failure the outputs
 *    and the context are unchanged, except for TSID_E_NONFINITE (see
 *    tsid_fit_template) and errors reported by tsid_sync.
 *  - TSID_E_DEVICE: a HIP call failed; tsid_last_error gives the detail.
 */
#ifndef TSID_H
#define TSID_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct tsid_ctx tsid_ctx;

typedef enum {
    TSID_OK = 0,
    TSID_E_INVAL = 1,     /* bad argument: NULL pointer, size < 0, unsupported k, bad option */
    TSID_E_RANGE = 2,     /* an index outside [0, m) / [0, n) / [0, n_fixed) / [0, n_free) */
    TSID_E_DUP = 3,       /* a repeated template id, or a repeated cell (Omega is a set) */
    TSID_E_NOMEM = 4,     /* device allocation failed or would exceed max_device_bytes */
    TSID_E_DEVICE = 5,    /* HIP runtime error */
    TSID_E_STATE = 6,     /* call out of order (e.g. fit before build) */
    TSID_E_NONFINITE = 7  /* a factor update produced Inf or NaN */
} tsid_status;

typedef enum { TSID_FP32 = 0, TSID_BF16 = 1 } tsid_precision;

/* Per-row step normalisation.  SUM: the plain full gradient of Eq. 2.
 * DEGREE: the step of every factor row is divided by max(1, its number of
 * observed cells) -- the 1/n normalisation of Eq. 5 (Section 5.1), applied to
 * both P and Q.  COL_DEGREE: the same division for the column factors Q only,
 * the rows of P taking the plain step, as Eq. 5 prints it (template fits
 * only; the extension returns E_INVAL). */
typedef enum { TSID_STEP_SUM = 0, TSID_STEP_DEGREE = 1, TSID_STEP_COL_DEGREE = 2 } tsid_step;

/* Fit options.
 *  epochs  number of full-gradient epochs (>= 0).
 *  lambda  l2 weight of Eq. 2 (>= 0).   lr  step size eta (> 0).
 *  clip    1: asymmetric clipping of Section 5.3 -- each coordinate of the
 *          row's summed descent direction, after the step scale of
 *          opts->step, becomes min(d, clip_xi) (positive components are
 *          capped, negative ones pass; NaN propagates).  clip_xi > 0.
 *          2: the same clip in the per-entry order (Section 5.3 applied to
 *          Eqs. 3-4 entry by entry, then the 1/n average of Eq. 5): each
 *          cell adds min(2 e q - 2 lambda p, clip_xi) per coordinate (the
 *          regulariser once per cell, the master p in it) and the row moves by
 *          lr times the sum (divided by its degree with the DEGREE step); a
 *          row without cells stays.  Template fits only, on the item pass
 *          (E_INVAL with TSID_PASS_SLAB or forced dense tiles; the automatic
 *          modes use neither); the extension returns E_INVAL.
 *          3: the clip of Section 5.3 in the order its printed update
 *          takes, the step scale s (1, or 1/max(1, deg) with a degree
 *          step) outside the min: each coordinate moves by
 *          lr * s * min(D, clip_xi), D the row's summed descent direction
 *          (clip 1 moves it by lr * min(s * D, clip_xi)).
 *          0: no clip.
 *  prec    TSID_FP32: fp32 factors.  TSID_BF16: the products read bf16
 *          (round-to-nearest-even) copies of the factors, accumulate in fp32,
 *          and an fp32 master copy takes the update (the mixed precision of
 *          Section 5.3, with bf16 in place of fp16).
 *  step    tsid_step. */
typedef struct {
    int32_t epochs;
    float lambda;
    float lr;
    float clip_xi;
    int32_t clip;
    int32_t prec;
    int32_t step;
} tsid_fit_opts;

/* Create a context on HIP device `device`.  hip_stream: a hipStream_t to run
 * the compute work on (for example torch's current stream), or NULL for a
 * stream owned by the context.  The context creates two more streams (host to
 * device copies, device to host copies), all at the default priority.
 * max_device_bytes: cap on the context's device allocations, 0 = no cap.
 * Errors: E_INVAL (out == NULL), E_DEVICE (bad device id or HIP failure). */
tsid_status tsid_create(int device, void *hip_stream, size_t max_device_bytes, tsid_ctx **out);

/* Release every resource of the context (waits for outstanding work first).
 * NULL is ignored. */
void tsid_destroy(tsid_ctx *ctx);

/* Detail of the last failure on this context (static storage owned by the
 * context; empty string if none). */
const char *tsid_last_error(const tsid_ctx *ctx);

/* Build the resident template (Section 3.2; Section 5.1 "Sampling the TSID
 * Template Submatrix"): template maps from I and J, the filter of Omega to
 * Omega* with local ids, and the buckets of Omega* by row (sorted by (a, b))
 * and by column (sorted by (b, a)).  Replaces any previous template.
 *  m, n          matrix shape (1 <= m, n < 2^31).
 *  u, i, r       HOST, nnz entries of Omega (COO).  Streamed to the device in
 *                pieces of stage_entries entries (0 = library default).
 *  I, J          HOST, m_t and n_t template ids (0 <= m_t <= m, 0 <= n_t <= n).
 *  k             rank; one of 8, 16, 32, 64, 128.
 * Errors: E_INVAL (NULL with a nonzero size, nnz < 0, bad k, non-finite r in
 * the template), E_RANGE (an id of I, J, u or i out of range), E_DUP (a
 * repeated id in I or J, or a cell (u, i) given twice anywhere in Omega:
 * when some cells fall outside the template, every cell's key is sorted on
 * the device, with 24 bytes per cell of temporary device memory), E_NOMEM,
 * E_DEVICE.  Synchronous. */
tsid_status tsid_build_template(tsid_ctx *ctx, int64_t m, int64_t n,
                                const int32_t *u, const int32_t *i, const float *r, int64_t nnz,
                                const int32_t *I, int32_t m_t, const int32_t *J, int32_t n_t,
                                int32_t k, int64_t stage_entries);

/* Sizes of the current template: rows m_t, columns n_t, |Omega*|, rank k.
 * Any output pointer may be NULL.  E_STATE before a build. */
tsid_status tsid_template_info(const tsid_ctx *ctx, int32_t *m_t, int32_t *n_t, int64_t *nnz,
                               int32_t *k);

/* Template fit (Stage I, Sections 3.2 and 5.1): opts->epochs full-gradient
 * epochs on the objective of Eq. 2 over Omega*,
 *   L(P, Q) = sum_(a,b) (r_ab - p_a . q_b)^2 + lambda (||P||_F^2 + ||Q||_F^2).
 * Epoch t computes every residual and both gradients (Eqs. 3-4) at (P_t, Q_t)
 * and moves every row of P and Q at once against its gradient (Eq. 5 with the
 * step of opts->step and the clip of opts->clip).  Each factor row is written
 * once per epoch by the unit that owns it; no atomic operations are used, and
 * the result is bitwise reproducible for a given pass kernel
 * (tsid_set_pass_kernel).
 *  P   DEVICE m_t x k: P_0 on entry, P_T on return.
 *  Q   DEVICE n_t x k: Q_0 on entry, Q_T on return.
 *  loss_hist  HOST epochs + 1 doubles or NULL: L(P_t, Q_t) for t = 0..epochs.
 * Errors: E_STATE (no template), E_INVAL (NULL factors with m_t or n_t > 0,
 * bad options), E_NOMEM, E_DEVICE, E_NONFINITE: some update of epoch t was not
 * finite; P and Q then hold P_t and Q_t (the last finite iterate), loss_hist
 * holds L for 0..t and NaN after.  Synchronous. */
tsid_status tsid_fit_template(tsid_ctx *ctx, float *P, float *Q, const tsid_fit_opts *opts,
                              double *loss_hist);

/* Epochs completed by the last tsid_fit_template on this context: opts->epochs
 * after success, t after TSID_E_NONFINITE (P and Q were returned at P_t, Q_t),
 * 0 before any fit.  Errors: E_INVAL (ctx or epochs NULL). */
tsid_status tsid_fit_epochs_done(const tsid_ctx *ctx, int32_t *epochs);

/* Objective of Eq. 2 over the template's Omega* at (P, Q) (DEVICE, fp32),
 * accumulated in fp64 in a fixed order.  With lambda = 0 it is the residual
 * sum of squares (used for held-out RMSE on a template built over test cells).
 * Errors: E_STATE, E_INVAL (NULL factors, out == NULL, lambda < 0), E_DEVICE.
 * Synchronous. */
tsid_status tsid_loss(tsid_ctx *ctx, const float *P, const float *Q, float lambda, double *out);

/* tsid_loss for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same value, bit for bit, computed by the same kernels, with every buffer
 * the kernels need (per-work-item residual sums, per-row norms, the
 * reduction's partial sums and result) taken from a fixed device array of
 * TSID_NOALLOC_SCRATCH_BYTES that the library's code object holds on each
 * device it runs on, until the process ends.  The call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine); the template and
 * its fp32 row-side work plan come from tsid_build_template.
 * Limit: 4 bytes per work item of the row side (at least one per template
 * row), 4 per template row and per template column, plus 2 KiB, must fit the
 * array (a 1 M x 100 k template with 4.2e8 cells needs about 9 MB).
 * Every call on a device shares that device's array: calls that overlap on
 * one device (several contexts, several host threads) race and must be
 * serialised by the caller.  Nothing in the array needs clearing between
 * calls (every slot a call reads is written by that call first).
 * Arguments, layout and errors as tsid_loss, plus E_NOMEM when the template
 * exceeds the limit (nothing is launched).  Synchronous. */
#define TSID_NOALLOC_SCRATCH_BYTES (32u << 20)
tsid_status tsid_loss_noalloc(tsid_ctx *ctx, const float *P, const float *Q, float lambda, double *out);

/* One chunk of the extension (Stage II, Section 5.2; Eq. 6 in factored form:
 * a free row's coefficients x_f solve the ridge problem
 *   min sum_(entries of f) (r - F_fixed[fixed_id] . x_f)^2 + lambda ||x_f||^2
 * with the fixed factors held constant).  Every free row starts at zero and
 * takes opts->epochs gradient steps of Eq. 5 (opts->step, opts->clip apply;
 * opts->prec is ignored: the fixed side is read in fp32).  A row's steps are
 * taken in one of two forms with the same result up to rounding:
 *  - per cell, with the template fit's residual/gradient kernel, in fp32,
 *    gathering the row's fixed factors once per step;
 *  - in Gram form, for rows of at least a threshold number of cells: the
 *    gradient 2 lambda x - 2 (b - G x) from G = sum p p^T and b = sum r p,
 *    accumulated once in fp64 on the matrix cores, with the steps in fp64.
 *    The threshold weighs the forms' work at this k and step count, and
 *    whether the fixed table fits one XCD's 4 MiB L2 (where the per-cell
 *    gathers are cheap): at 20 steps, from 40 (k = 32) or never (k = 64)
 *    cells with such a table, and from 69 (k = 32) or 96 (k = 64) cells
 *    with a larger one.  k = 128 and a single step keep the per-cell form.
 *    A row's form depends on its own cell count only, so results do not
 *    depend on how the rows are split into chunks.
 * The chunk's cells are bucketed by free row on the device (a stable sort by
 * (free_local, fixed_id)); cells that already come in that order (as a
 * line-by-line generator emits them) skip the sort, with the same result.
 *  side        0: the free rows are rows of R and F_fixed holds column
 *              factors; 1: the free rows are columns and F_fixed holds row
 *              factors.  The arithmetic is the same; side is recorded only.
 *  fixed_id    HOST nnz ids into F_fixed (0 <= id < n_fixed).
 *  free_local  HOST nnz ids of the free rows (0 <= f < n_free).
 *  r           HOST nnz values.
 *  F_fixed     DEVICE n_fixed x k (k of the current template), read only;
 *              must stay unchanged until the chunk completes.
 *  F_free      n_free x k, written when the chunk completes: host memory
 *              (pinned, for the copies to overlap), or device memory of the
 *              context's device, where the results are copied on the device
 *              (a caller that feeds them to a later phase keeps them in HBM).
 * Asynchronous: the chunk's host-to-device copy runs on the context's copy
 * stream while the previous chunk computes, and the results return on a third
 * stream (Section 5.2, double-buffered pipelining); two device staging slots
 * alternate between consecutive chunks.  The call returns once the previous
 * chunk's host-to-device copy has finished: from then on that chunk's host
 * input arrays (fixed_id, free_local, r) are no longer read and may be
 * refilled, so a caller can stream chunks through two pinned host buffers.
 * Every other host buffer (this chunk's inputs, every F_free) must stay valid
 * until tsid_sync returns, which also writes the last F_free.  Pinned host
 * memory is needed for the copies to overlap.
 * Errors returned here: E_STATE (no template: k unknown), E_INVAL, E_NOMEM,
 * E_DEVICE.  Errors found on the device (E_RANGE for ids out of range, E_DUP
 * for a repeated (fixed_id, free_local) cell, E_NONFINITE) are returned by the
 * next tsid_sync; the affected chunk's F_free is then unspecified. */
tsid_status tsid_extend_chunk(tsid_ctx *ctx, int side, const int32_t *fixed_id,
                              const int32_t *free_local, const float *r, int64_t nnz,
                              int32_t n_free, const float *F_fixed, int64_t n_fixed,
                              float *F_free, const tsid_fit_opts *opts);

/* One chunk of the extension solved exactly (Stage II, Section 5.2; Eq. 6 in
 * factored form, the alternating-least-squares step): each free row is the
 * ridge regression
 *   x_f = (sum_(entries of f) p p^T + lambda I)^{-1} sum_(entries of f) r p,
 * p = F_fixed[fixed_id], the minimiser that tsid_extend_chunk's gradient
 * steps approach.  The Gram matrices are accumulated on the matrix cores in
 * fp64 (v_mfma_f64_16x16x4f64) and each is factored (Cholesky) and solved in
 * fp64, by one wavefront for k <= 64 (the matrix in registers) and by a
 * workgroup of four wavefronts for k = 128 (the matrix in 130 KiB of LDS);
 * F_free receives the fp32 rounding of the solution.
 * A free row without entries gets x_f = 0.
 * Arguments, layout, ownership, asynchrony and the staging slots are those of
 * tsid_extend_chunk; lambda >= 0 replaces the options.
 * Errors returned here: E_STATE (no template), E_INVAL (bad sizes or
 * pointers, lambda negative or not finite, k not in {8, 16, 32, 64, 128}), E_NOMEM,
 * E_DEVICE.  At the next tsid_sync: E_RANGE / E_DUP as for tsid_extend_chunk,
 * and E_NONFINITE when a Gram matrix is not positive definite (lambda = 0 and
 * fewer independent entries than k in some row) or a solution is not finite;
 * the affected chunk's F_free is then unspecified. */
tsid_status tsid_extend_chunk_ridge(tsid_ctx *ctx, int side, const int32_t *fixed_id,
                                    const int32_t *free_local, const float *r, int64_t nnz,
                                    int32_t n_free, const float *F_fixed, int64_t n_fixed,
                                    float *F_free, float lambda);

/* One chunk of the extension as Eq. 6 states it (Stage II, Section 5.2):
 * free line f is represented in the fixed template basis by a coefficient
 * vector c_f with one entry per basis line, its entries are predicted as
 * p . (B^T c_f) with p = F_fixed[fixed_id] (R* = P B^T in factored form), and
 *   L(C) = sum_(entries) (r - p . B^T c_f)^2 + lambda ||C||_F^2
 * is minimised by the Adam method from C = 0 for opts->steps steps: per step
 * the gradient G = dL/dC, m <- beta1 m + (1 - beta1) G,
 * w <- beta2 w + (1 - beta2) G^2, and C <- C - lr m^ / (sqrt(w^) + eps) with
 * the bias corrections m^ = m / (1 - beta1^t), w^ = w / (1 - beta2^t) at step
 * t = 1, 2, ...  All arithmetic is fp32 on the device; every sum has a fixed
 * order.
 *  basis     DEVICE n_basis x k fp32 (the template's factors of the side the
 *            coefficients span: Q_J for free columns, P_I for free rows),
 *            16-byte aligned; must stay unchanged until the chunk completes.
 *  F_free    HOST n_free x k: receives B^T c_f after the last step.
 *  C_out     HOST n_free x n_basis, or NULL: receives C.
 * The other arguments, asynchrony and staging are those of tsid_extend_chunk;
 * device memory per staging slot grows by 12 n_free n_basis bytes.
 * Errors returned here: E_STATE (no template), E_INVAL (bad sizes or
 * pointers, steps < 0, lambda or eps negative or not finite, lr not finite,
 * beta1 or beta2 outside [0, 1), k not in {8, 16, 32, 64, 128}), E_NOMEM,
 * E_DEVICE.  At the next tsid_sync: E_RANGE / E_DUP as for
 * tsid_extend_chunk, E_NONFINITE if a coefficient becomes non-finite. */
typedef struct {
    int32_t steps;
    float lambda, lr, beta1, beta2, eps;
} tsid_adam_opts;
tsid_status tsid_extend_chunk_adam(tsid_ctx *ctx, int side, const int32_t *fixed_id,
                                   const int32_t *free_local, const float *r, int64_t nnz,
                                   int32_t n_free, const float *F_fixed, int64_t n_fixed,
                                   const float *basis, int64_t n_basis, float *F_free,
                                   float *C_out, const tsid_adam_opts *opts);

/* Wait for every outstanding chunk; returns the first device-side error of
 * those chunks (and clears it), else TSID_OK. */
tsid_status tsid_sync(tsid_ctx *ctx);

/* Kernel that runs the P and Q passes of tsid_fit_template (the arithmetic is
 * the same; the mapping onto the GPU differs).
 *  TSID_PASS_ITEM  every bucket is cut into work items of a few hundred cells,
 *                  each taken by a group of lanes that gathers the other
 *                  factor's rows from the cache hierarchy.  Any rank,
 *                  precision and degree distribution.
 *  TSID_PASS_SLAB  one lane per factor row; the other factor is staged
 *                  through LDS in 128 KiB slabs shared by a block of 512 rows.
 *                  fp32 factors with k in {8, 16, 32, 64}; fastest when the
 *                  cells are spread evenly (uniformly sampled templates).
 *  TSID_PASS_AUTO  (default) the slab pass for a side whose template is fp32,
 *                  k <= 64, holds on average at least 4 cells per staged row
 *                  and block of 512 rows, and has no bucket longer than twice
 *                  the mean plus 64; the item pass otherwise.
 * Takes effect at the next tsid_fit_template.  Errors: E_INVAL (unknown mode);
 * a fit with TSID_PASS_SLAB on an unsupported rank or precision returns
 * E_INVAL. */
enum { TSID_PASS_AUTO = 0, TSID_PASS_ITEM = 1, TSID_PASS_SLAB = 2 };
tsid_status tsid_set_pass_kernel(tsid_ctx *ctx, int mode);

/* Pass kernels the last tsid_fit_template ran (TSID_PASS_ITEM or
 * TSID_PASS_SLAB) for the P pass and the Q pass; 0 before any fit.  Either
 * output may be NULL.  Errors: E_INVAL (ctx NULL). */
tsid_status tsid_fit_pass_kernels(const tsid_ctx *ctx, int32_t *p_pass, int32_t *q_pass);

/* Dense head tiles for bf16 fits (Eqs. 2-4 evaluated on the matrix cores).
 * The template's cells are grouped into 16 x 16 tiles of the (row, column)
 * grid; a tile holding at least fill * 256 cells is handled by a
 * matrix-core kernel: with the tile's residuals E (zero at unobserved
 * cells), the row-side gradient sums E Q_J and the column-side sums E^T P_I
 * are products of a 16 x 16 tile and a 16 x k slab of factors, computed
 * with bf16 inputs and fp32 accumulation (the residual is split into a
 * bf16 high part and a bf16 remainder, so its fp32 value enters the
 * product to about 2^-16 relative).  The item pass then walks only the
 * remaining cells and adds the tile sums before the update.  The epochs are
 * the same; rounding differs from the all-item path at the level of the
 * bf16 factors (Section 5.3).
 *  fill < 0   (default) automatic: fill 0.15 (0.10 at k = 128), used
 *             when bf16, k in {16, 32, 64, 128}, and the dense tiles hold
 *             at least 10% of the cells.
 *  fill = 0   off.
 *  0 < fill <= 1  forced with this fill threshold (bf16 fits with k in
 *             {16, 32, 64, 128}; other fits return E_INVAL).
 * The tiles are laid out at the first bf16 fit after a template or mode
 * change and kept with the template: 1 KiB of device memory per dense tile
 * and side (its values, fp32, NaN at unobserved cells), the other cells'
 * streams (8 bytes per cell and side) and a rows x k fp32 buffer of tile
 * sums per side.  Takes effect at the next tsid_fit_template.
 * Errors: E_INVAL (ctx NULL, fill > 1 or NaN). */
tsid_status tsid_set_dense_tiles(tsid_ctx *ctx, float fill);

/* What the last tsid_fit_template handled as dense tiles (all zero when it
 * used none): cells in dense tiles, dense tiles, and the 16-row stripes of
 * the P pass (stripes[0], rows of the template) and of the Q pass
 * (stripes[1], columns) that hold at least one dense tile.
 * Errors: E_INVAL (ctx or out NULL). */
typedef struct {
    int64_t cells;
    int64_t tiles;
    int64_t stripes[2];
} tsid_dense_info;
tsid_status tsid_fit_dense_info(const tsid_ctx *ctx, tsid_dense_info *out);

/* Multi-view similarity term for tsid_fit_template (Section 5.1: the
 * item-factor update with the similarity regulariser of Eq. 1, the item
 * similarity S of Section 2.2 given here as a sparse matrix).  S is over the
 * template's columns (ids are positions in J), symmetric, with both
 * orientations of every off-diagonal entry listed once (HOST COO row, col,
 * val; nnz entries; values finite and >= 0; diagonal entries allowed, they
 * add nothing).  The objective of Eq. 2 gains
 *   (beta / 2) sum_(i, i') S_ii' ||q_i - q_i'||^2,
 * whose gradient with respect to q_i, 2 beta sum_i' S_ii' (q_i - q_i'), is the
 * update's similarity term: every epoch it is evaluated at Q_t (the fp32
 * master) and joins q_i's summed gradient before the step rule and the clip
 * (opts->clip 0 or 1); the loss history includes the term.  The fits then
 * run the item pass on both sides (dense tiles allowed): a fit with
 * TSID_PASS_SLAB, clip 2 or mini-batch epochs returns E_INVAL.  tsid_loss
 * stays Eq. 2.  S is copied to the device (CSR, 12 bytes per entry, plus 4k
 * bytes per column for the gradient sums) and kept with the template until
 * the next call or template; nnz = 0 or beta = 0 turns the term off.
 * Errors: E_STATE (no template), E_INVAL (NULL arrays with nnz > 0, nnz < 0,
 * beta negative or not finite, a value negative or not finite, S not
 * symmetric), E_RANGE (an id outside [0, n_t)), E_DUP (a repeated entry),
 * E_NOMEM, E_DEVICE. */
tsid_status tsid_set_similarity(tsid_ctx *ctx, const int32_t *row, const int32_t *col, const float *val,
                                int64_t nnz, float beta);

/* Mini-batch epochs for tsid_fit_template (Section 5.1: the stochastic
 * method updates the factors within an epoch, Eq. 5 averaging each update
 * over the entries it uses; here the entries are grouped into mini-batches).
 * Cell (a, b) of the template (a: position of its row in I, b: of its column
 * in J) belongs to batch splitmix64(seed ^ (a << 32 | b)) mod n_batches, with
 * splitmix64 the output function of the SplitMix64 generator (Steele, Lea and
 * Flood, 2014).  Each epoch then takes one step per batch, in batch order:
 * the Jacobi step of Eqs. 3-5 (with the options' step rule and clip) on the
 * batch's cells only, from the factors the previous batch left, where the
 * degree step divides by the line's cell count in the batch and rows and
 * columns without a cell in the batch keep their values.  The loss history
 * holds L(P, Q) over every cell at the start of each epoch and after the
 * last.  On a non-finite update the fit returns E_NONFINITE with the factors
 * before the failing batch step; tsid_fit_epochs_done gives the whole epochs
 * completed before it, and the loss entries of later epochs are NaN.
 *  n_batches = 0   (default) full-gradient (Jacobi) epochs.
 *  1 <= n_batches <= TSID_MAX_BATCHES   mini-batch epochs; they run the item
 *                  pass (a fit with TSID_PASS_SLAB or forced dense tiles
 *                  returns E_INVAL), and n_batches times the template's rows
 *                  (and columns) must be below 2^31.
 * The batch-major copies of the streams (8 bytes per cell and side) and the
 * batch pointers (8 bytes per batch and row or column) are built at the
 * first such fit after a template, batch-count or seed change and kept with
 * the template.  With timing on, pass_ms / fixup_ms cover the first batch's
 * passes of a timed epoch and epoch_ms the whole epoch (its loss pass
 * included).  Takes effect at the next tsid_fit_template.
 * Errors: E_INVAL (ctx NULL, n_batches outside [0, TSID_MAX_BATCHES]). */
#define TSID_MAX_BATCHES 4096
tsid_status tsid_set_minibatch(tsid_ctx *ctx, int32_t n_batches, uint64_t seed);

/* Row-blocked Q passes of the item pass.  The Q pass gathers a row of P for
 * every cell; when P's table (m_t x k, bf16 or fp32) is larger than the
 * last-level cache those gathers go to HBM and the cache hierarchy's miss
 * bandwidth bounds the pass.  With n blocks, the rows of P are cut into n
 * ranges holding about equal shares of the Q pass's cells; every column's
 * cells whose row falls in block j form one work bucket, all blocks run in
 * one launch, and the workgroups of each group of 8 blocks are dealt in turn
 * to the device's 8 XCDs, so that each XCD gathers from its own block; the
 * groups pair the blocks from both ends of P (0, n - 1, 1, n - 2, ...), so
 * that every group gathers from about the same share of the table.  Each
 * bucket stores its partial gradient sum
 * (n x n_t x k fp32 of device memory); a second kernel adds the n sums of a
 * column in block order and updates it.  The arithmetic is the same; the fp32
 * sums of a column are added in another order.
 *  n_blocks = 0  (default) automatic: blocks of about 11 MiB of P, their
 *                count rounded up to a multiple of 8, when the table exceeds
 *                96 MiB (Billion-scale: 24 blocks), else one.
 *  n_blocks = 1  off.   2 <= n_blocks <= TSID_MAX_ROW_BLOCKS: forced.
 * Applies to full-gradient fits whose Q pass runs the item pass.  Takes effect
 * at the next tsid_fit_template.  Errors: E_INVAL (ctx NULL, n_blocks out of
 * range). */
#define TSID_MAX_ROW_BLOCKS 64
tsid_status tsid_set_row_blocks(tsid_ctx *ctx, int32_t n_blocks);
/* Row blocks the last tsid_fit_template's Q pass ran with (1: one pass).
 * Errors: E_INVAL (ctx or n_blocks NULL). */
tsid_status tsid_fit_row_blocks(const tsid_ctx *ctx, int32_t *n_blocks);

/* Kernel timing of the template fit (a tracing aid).  With every = n > 0,
 * the kernels of every n-th epoch of tsid_fit_template (epochs 0, n, 2n, ...)
 * are launched with a start and an end HIP event attached to their dispatch
 * on the compute stream (no separate event packets), and so is every loss
 * reduction; the durations accumulate here until the next tsid_set_timing
 * call resets them.  Each timed dispatch costs a few microseconds of wall
 * time, so timing a sample of the epochs keeps the fit's own throughput
 * nearly unchanged.  every = 0 turns timing off.
 *  pass_ms[0] / pass_launches[0]: the P pass (row buckets); [1]: the Q pass
 *  (column buckets).  The two passes of an epoch go out as one launch,
 *  counted in [0] ([1] stays 0), unless the Q pass runs in row blocks
 *  (tsid_set_row_blocks); the slab pass's two finishing kernels are then one
 *  launch too, counted once under fixup.  fixup: the kernels that combine
 *  partial sums after a pass (item pass: buckets longer than one wave; slab pass: blocks split
 *  over several workgroups), which also update those rows; reduce: the
 *  batched loss reductions (one per 16 epochs); dense_ms[0] / [1]: the
 *  dense-tile kernels before the P / Q pass (tsid_set_dense_tiles); when
 *  the passes share a launch, both sides' tiles share one too, counted in
 *  [0];
 *  epoch_ms: from the start of a timed epoch's first kernel to the end of
 *  its last, summed over the timed epochs, whose number is `epochs`;
 *  ext_h2d_ms / ext_compute_ms / ext_chunks: for the extension chunks queued
 *  while timing is on (every chunk, whatever `every`), the host-to-device
 *  copy of each chunk on the copy stream and its compute on the compute
 *  stream (bucketing and solve), summed, and the chunk count; a chunk is
 *  counted once the slot it used is reused or at tsid_sync.
 * Errors: E_INVAL (ctx NULL or every < 0). */
typedef struct {
    double pass_ms[2];
    int64_t pass_launches[2];
    double fixup_ms;
    int64_t fixup_launches;
    double reduce_ms;
    int64_t reduce_launches;
    double epoch_ms;
    int64_t epochs;
    double dense_ms[2];
    int64_t dense_launches[2];
    double ext_h2d_ms;
    double ext_compute_ms;
    int64_t ext_chunks;
} tsid_timing;
tsid_status tsid_set_timing(tsid_ctx *ctx, int every);
tsid_status tsid_get_timing(const tsid_ctx *ctx, tsid_timing *out);

/* Index structures of the current template, copied to host_dst (HOST) for
 * bit-exact checks.  which / element type / count:
 *   TSID_IDX_ROW_MAP int32 m      TSID_IDX_COL_MAP int32 n
 *   TSID_IDX_ROW_PTR int64 m_t+1  TSID_IDX_CSR_COL int32 nnz  TSID_IDX_CSR_VAL fp32 nnz
 *   TSID_IDX_COL_PTR int64 n_t+1  TSID_IDX_CSC_ROW int32 nnz  TSID_IDX_CSC_VAL fp32 nnz
 *   TSID_IDX_DEG_R   int32 m_t    TSID_IDX_DEG_C   int32 n_t
 *   TSID_IDX_BATCH_PTR_R int64 B*m_t+1   TSID_IDX_BATCH_PTR_C int64 B*n_t+1
 * The batch pointers (after a mini-batch fit, B its batch count; E_STATE
 * before): entry beta * rows + x is the first cell of row (column) x of
 * batch beta in the batch-major stream, so the cells of row x in batch beta
 * number ptr[beta * m_t + x + 1] - ptr[beta * m_t + x].
 * bytes must equal count * element size.  Errors: E_STATE, E_INVAL, E_DEVICE. */
enum {
    TSID_IDX_ROW_MAP = 0, TSID_IDX_COL_MAP = 1, TSID_IDX_ROW_PTR = 2, TSID_IDX_CSR_COL = 3,
    TSID_IDX_CSR_VAL = 4, TSID_IDX_COL_PTR = 5, TSID_IDX_CSC_ROW = 6, TSID_IDX_CSC_VAL = 7,
    TSID_IDX_DEG_R = 8, TSID_IDX_DEG_C = 9, TSID_IDX_BATCH_PTR_R = 10, TSID_IDX_BATCH_PTR_C = 11
};
tsid_status tsid_export_index(const tsid_ctx *ctx, int which, void *host_dst, size_t bytes);

/* Chunk partition of the free rows (Section 5.2: the matrix is split into
 * chunks of whole rows/columns processed independently).  Host-only, needs no
 * context or device.  counts[f] (HOST, n_free values >= 0) = observed cells
 * of free row f, in order.
 *  n_chunks > 0: exactly n_chunks contiguous runs (some may be empty); run j
 *    starts at the first f that has at least ceil(j * total / n_chunks) cells
 *    in the rows before it.
 *  n_chunks == 0: greedy runs of at most max_entries cells (> 0); a single
 *    row above the cap forms its own run.
 * bounds (HOST, max_bounds entries) receives the start of every run followed
 * by n_free.  Returns the number of runs, or -1 on a bad argument or when
 * max_bounds is too small. */
int32_t tsid_chunk_plan(const int64_t *counts, int64_t n_free, int32_t n_chunks,
                        int64_t max_entries, int64_t *bounds, int32_t max_bounds);

#ifdef __cplusplus
}
#endif

#endif /* TSID_H */
