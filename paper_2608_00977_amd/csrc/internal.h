// Internal declarations of libtsid (not part of the public C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "tsid.h"

namespace tsid {

// Failures inside the library are thrown as this and mapped to a status at
// the C boundary.
struct Error {
    tsid_status st;
    std::string msg;
};

[[noreturn]] void fail(tsid_status st, const std::string &msg);
void hip_check(hipError_t e, const char *what);
#define TSID_HIP(expr) ::tsid::hip_check((expr), #expr)

// Device-side error slots (plain stores of 1, never atomics).
enum ErrSlot { ERR_RANGE = 0, ERR_DUP = 1, ERR_INVAL = 2, ERR_NONFINITE = 3, ERR_SLOTS = 4 };

// Step of one coordinate of a factor row (Eq. 5 with the Section 5.3 clip):
// g is the summed gradient (Eqs. 3-4 over the row's cells plus the
// regulariser once), s the step scale of the row (1 or 1/max(1, deg)).  The
// descent direction is -g.  clip 0: s (-g); clip 1: min(s (-g), xi), the clip
// on the normalised direction; clip 3: s min(-g, xi), the clip before the
// scale, in the order the clipped update of Section 5.3 prints.  A NaN
// compares false and passes through.
__device__ __forceinline__ float clipped_step(float g, float s, int32_t clip, float xi) {
    if (clip == 3) {
        float d = -g;
        if (d > xi) d = xi;
        return s * d;
    }
    float d = -s * g;
    if (clip && d > xi) d = xi;
    return d;
}

inline int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }
inline int bits_for(int64_t count) {  // bits to hold values 0..count-1 (at least 1)
    int b = 1;
    while (b < 63 && (int64_t(1) << b) < count) ++b;
    return b;
}

// ------------------------------------------------------------ primitives
// Exclusive prefix sum of n uint32 values (in == out allowed).  If total is
// non-null the grand total is stored there (device).  `scratch` must hold
// scan_scratch_elems(n) uint32.
size_t scan_scratch_elems(int64_t n);
void scan_u32(const uint32_t *in, uint32_t *out, int64_t n, uint32_t *total, uint32_t *scratch,
              hipStream_t s);

// Stable LSD radix sort of (key, value) pairs on the low `nbits` bits of the
// key, 8 bits per pass.  Ping-pongs between the two buffers; returns true if
// the sorted result ends in the *_alt buffers.  scratch: radix_scratch_elems(n).
// unsorted (device, or null): a flag from keys_unsorted; when it holds 0 the
// input is already in key order and the passes only leave it in the buffer
// the return value names.
size_t radix_scratch_elems(int64_t n);
bool radix_sort(uint64_t *keys, uint32_t *vals, uint64_t *keys_alt, uint32_t *vals_alt, int64_t n,
                int nbits, uint32_t *scratch, hipStream_t s, const uint32_t *unsorted = nullptr);
// *unsorted = 1 if some key is smaller than the one before it, else 0.
void keys_unsorted(const uint64_t *keys, int64_t n, uint32_t *unsorted, hipStream_t s);

void fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s);
void fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t s);
void fill_f32(float *p, int64_t n, float v, hipStream_t s);
void scatter_map(const int32_t *ids, int32_t count, int32_t *map, hipStream_t s);

// Filter of one staging piece of Omega to the template (order preserving).
// Writes packed keys (a << bits_b | b) and value bits at out + base.
// bcnt/boffs: filter_blocks(S) uint32 each; piece_total: 1 uint32 (device).
int filter_blocks(int64_t S);
void filter_count(const int32_t *u, const int32_t *i, const float *r, int64_t S,
                  const int32_t *row_map, const int32_t *col_map, int64_t m, int64_t n,
                  uint32_t *bcnt, int32_t *err, hipStream_t s);
void filter_write(const int32_t *u, const int32_t *i, const float *r, int64_t S,
                  const int32_t *row_map, const int32_t *col_map, int64_t m, int64_t n,
                  const uint32_t *boffs, int64_t base, int bits_b, uint64_t *out_key,
                  uint32_t *out_val, hipStream_t s);

// After a sort on packed keys: stream[j] = {key & low_mask, value}; flags a
// repeated key as ERR_DUP.
// keys[j] = u[j] * n + i[j] (and vals[j] = 0) for a piece of Omega.
void cell_keys(const int32_t *u, const int32_t *i, int64_t len, int64_t n, uint64_t *keys, uint32_t *vals,
               hipStream_t s);
// err[ERR_DUP] = 1 if two neighbours of the sorted keys are equal.
void adjacent_equal(const uint64_t *keys, int64_t n, int32_t *err, hipStream_t s);
void keys_to_stream(const uint64_t *keys, const uint32_t *vals, int64_t n, int low_bits,
                    int2 *stream, int32_t *err, hipStream_t s);
// ptr[x] = first position whose key >> low_bits >= x, for x in [0, rows].
void ptr_from_keys(const uint64_t *keys, int64_t n, int32_t rows, int low_bits, int64_t *ptr,
                   hipStream_t s);
// (hi << lo_bits | lo) -> (lo << hi_bits | hi).
void swap_key_halves(const uint64_t *keys, int64_t n, int lo_bits, int hi_bits, uint64_t *out,
                     hipStream_t s);
// Extension chunk keys: key = free << bits_fixed | fixed; out-of-range ids -> ERR_RANGE.
void chunk_keys(const int32_t *fixed_id, const int32_t *free_id, const float *r, int64_t nnz,
                int64_t n_fixed, int32_t n_free, int bits_fixed, uint64_t *keys, uint32_t *vals,
                int32_t *err, hipStream_t s);

// Work plan of a bucketed stream: every bucket (row) becomes
// max(1, ceil(deg / E)) items of at most E entries.  item_off has rows + 1
// entries (item_off[rows] = total items); items[j] = bucket of item j.
// nparts_scratch: rows uint32; scan_scratch: scan_scratch_elems(rows).
void plan_items(const int64_t *ptr, int32_t rows, int32_t E, uint32_t *item_off, int32_t *items,
                uint32_t *nparts_scratch, uint32_t *scan_scratch, hipStream_t s);

// Mini-batch epochs (minibatch.hip): keys[j] = batch * rows + owner row of
// cell j of a bucketed stream (side 0: rows of the template, side 1: its
// columns) and vals[j] = j; then out[j] = in[idx[j]].
void batch_keys(const int2 *stream, const int64_t *ptr, int32_t rows, int side, uint64_t seed, int32_t n_batches,
                uint64_t *keys, uint32_t *vals, hipStream_t s);
void gather_stream(const int2 *in, const uint32_t *idx, int64_t n, int2 *out, hipStream_t s);

// ------------------------------------------------------------------- fit
struct PassArgs {
    const int2 *stream;      // bucketed entries {other id, value bits}
    const int64_t *ptr;      // bucket pointers (rows + 1)
    const int32_t *items;    // bucket of each item (-1: an idle pad item)
    const uint32_t *item_off;  // first item of each bucket
    const uint32_t *item_end;  // one past the last item of each bucket
    const uint32_t *n_items_dev;  // device item count (or null: use n_items)
    int32_t n_items;         // item count, or an upper bound when n_items_dev is set
    int32_t rows;            // buckets
    int32_t E;               // entries per item
    const float *X;          // owner factors, fp32 master (rows x K)
    const void *Y;           // gathered factors: fp32, or bf16 bits in bf16 mode
    int64_t y_rows;          // rows of Y (bounds of the gathers)
    float *Xn;               // updated owner factors (null in loss-only mode)
    uint16_t *Xn_b;          // bf16 copy of Xn (bf16 mode) or null
    float *carry;            // partial gradient sums of split buckets (n_items x K)
    float *e2;               // per-item residual sum of squares, or null
    float *norm;             // per-row ||x||^2 of the owner rows, or null
    float lam, lr, xi;
    int32_t clip, degree;
    int32_t *err;            // device error slots
    int32_t epoch;           // a non-finite update stores epoch + 1 in err[ERR_NONFINITE]
    int32_t skip_after_nonfinite;  // 1: do nothing if an earlier epoch stored a flag
    // With dense head tiles (bf16): the stream holds the cells outside them,
    // dptr gives each bucket's full degree (for the degree step), and gd the
    // dense cells' gradient sums of the rows whose 16-row stripe has dense
    // tiles (gd_tile_ptr[st + 1] > gd_tile_ptr[st]), added before the update.
    const int64_t *dptr;     // or null: degrees from ptr
    const float *gd;         // rows x K, or null
    const uint32_t *gd_tile_ptr;
    // 1: a bucket without cells keeps its row as it is (a mini-batch step
    // touches only the rows and columns of the batch's cells)
    int32_t keep_empty;
    // rows x K extra gradient added (times gx_scale) before the update, or null
    const float *gx;
    float gx_scale;
    // Row-blocked passes: bucket x spans ptr[x] .. ptr_end[x] (null: ptr[x + 1]),
    // and with partial_out the pass stores each bucket's gradient sum there
    // (rows x K) instead of updating the row.
    const int64_t *ptr_end;
    float *partial_out;
    // Row-blocked passes in one launch: buckets are (block, owner) pairs
    // v = block * owner_mod + owner, so the owner row is v % owner_mod (0: the
    // bucket is the owner row).
    int32_t owner_mod;
    // 1: the partial sum a wave leaves for a bucket longer than one wave sits
    // at carry + (item / groups per wave) * K, one per wave (plans built on
    // the host, whose longer buckets fill whole waves); 0: at carry + item * K.
    int32_t carry_per_wave;
    // Extension steps: free rows with at least this many cells are left to
    // the Gram-form kernel (0: none).
    int64_t skip_from;
};

// prec: 0 fp32, 1 bf16.  loss_only: residuals, e2 and norms only.
// ev0 / ev1 (may be null): HIP events that take the kernel's own start and end
// timestamps (attached to its dispatch; no extra packets on the stream).
// The item pass over a plan laid out in workgroup-sized chunks: workgroup w
// runs the chunk sched[w] (its first item / (waves * groups per wave)), or
// nothing when sched[w] < 0.  Not for loss-only passes.
void launch_item_pass_sched(int K, int prec, const PassArgs &a, const int32_t *sched, int64_t n_wg, hipStream_t s,
                            hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// Items of one workgroup of the item pass (waves per workgroup x groups per wave).
int items_per_workgroup(int K, int prec);
void launch_item_pass(int K, int prec, bool loss_only, const PassArgs &a, hipStream_t s,
                      hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// The P pass (a0) and the Q pass (a1) of one simultaneous step in one launch
// (full-gradient, not loss-only; two launches if the sides' gathers differ).
void launch_item_pass_pair(int K, int prec, const PassArgs &a0, const PassArgs &a1, hipStream_t s,
                           hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
void launch_fixup(int K, int prec, const PassArgs &a, hipStream_t s, hipEvent_t ev0 = nullptr,
                  hipEvent_t ev1 = nullptr);
// Row blocks of a bucketed stream: bounds[j * rows + x] = first cell of bucket
// x whose other index is >= row_bounds[j], for j = 0 .. n_blocks (int64;
// row_bounds holds n_blocks + 1 nondecreasing device values).
void launch_block_bounds(const int2 *stream, const int64_t *ptr, int32_t rows, int32_t n_blocks,
                         const int64_t *row_bounds, int64_t *bounds, hipStream_t s);
// After the n_blocks partial passes: row x's sums part[j * rows * K + x * K ..]
// added in block order, then the row update of `a` (its own bucket pointers
// give the degrees).
void launch_block_combine(int K, int prec, const PassArgs &a, const float *part, int32_t n_blocks, hipStream_t s,
                          hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
// `steps` one-sided extension steps from zero in one launch, one wave per
// bucket (a.rows buckets over a.stream / a.ptr; fp32; a.X unused, the result
// goes to a.Xn; a non-finite update stores 1 in a.err[ERR_NONFINITE]).
void launch_extend_steps(int K, const PassArgs &a, int32_t steps, hipStream_t s);
// Items one wave holds for rank K and precision prec (the item pass's groups
// per wave): buckets whose items stay inside one such run need no fixup.
int items_per_wave(int K, int prec);
void launch_row_norms(int K, const float *X, int32_t rows, float *norm, hipStream_t s);
void launch_to_bf16(const float *X, int64_t n, uint16_t *Xb, hipStream_t s);
// Loss of n_slots epochs at once: slot j holds e2 + j * e2_stride (ne per-item
// squared residual sums), np + j * nnp and nq + j * nnq (row norms), and
// out[j] = S_e + lam (S_p + S_q), each S a fixed-order fp64 sum, plus
// w4 S_s over ns + j * nns when ns is given (the similarity term).  With err,
// a slot whose epoch (epoch0 + j) follows a non-finite update is left
// unwritten.  partial: reduce_scratch_elems(n_slots) doubles.
size_t reduce_scratch_elems(int n_slots);
void launch_loss_reduce(const float *e2, int64_t e2_stride, int64_t ne, const float *np, int64_t nnp,
                        const float *nq, int64_t nnq, double lam, int n_slots, double *partial,
                        double *out, const int32_t *err, int32_t epoch0, hipStream_t s,
                        hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr, const float *ns = nullptr,
                        int64_t nns = 0, double w4 = 0.0);

// Multi-view similarity term (similarity.hip): for every template column i,
// gs[i] = sum_e S_e (q_i - q_col[e]) and se[i] = sum_e S_e ||q_i - q_col[e]||^2
// over the entries e of row i of S (CSR ptr / col / val), from fp32 Q.  se
// may be null.
void launch_sim_terms(int K, const int64_t *ptr, const int32_t *col, const float *val, int32_t n, const float *Q,
                      float *gs, float *se, hipStream_t s);

// ------------------------------------------------------------- slab pass
// Owner rows per workgroup (one lane each) and LDS bytes of one slab of the
// gathered factor.
#ifndef TSID_SLAB_LANES
#define TSID_SLAB_LANES 512
#endif
#ifndef TSID_SLAB_KIB
#define TSID_SLAB_KIB 128
#endif
constexpr int kSlabLanes = TSID_SLAB_LANES;
constexpr int kSlabBytes = TSID_SLAB_KIB * 1024;

struct SlabArgs {
    // The pass's own copy of the cells (launch_slab_order): for each slab s
    // and bucket x (slab-major: all runs of slab 0, then slab 1, ...) the
    // bucket's cells whose other id lies in the slab, padded to a multiple
    // of 8 records.  Records j = 8 g .. 8 g + 7 form block g of 48 bytes,
    // sblk[3 g .. 3 g + 2]: their rows within the slab (other id - s * C,
    // 16 bits each; C for a pad, the zero row the pass keeps after the slab
    // in LDS), then their values (fp32; 0 for a pad).
    const uint4 *sblk;
    const uint32_t *seg;     // seg[s * rows + x]: first record of run (x, s); seg[n_slabs * rows]: total
    const int64_t *ptr;      // bucket pointers of the template (a row's degree)
    int32_t rows;            // owner rows (buckets)
    int32_t y_rows;          // rows of the gathered factor
    int32_t C;               // gathered rows per slab
    int32_t n_slabs;         // ceil(y_rows / C)
    int32_t slabs_per_unit;  // S: slabs one workgroup walks
    int32_t units_per_block; // U = ceil(n_slabs / S): workgroups per block of kSlabLanes rows
    const float *X;          // owner factors (rows x K)
    const float *Y;          // gathered factors (y_rows x K)
    float *Xn;               // updated owner factors
    float *carry;            // partial sums, [units][kSlabLanes][K] (U > 1)
    float *e2;               // per-lane residual sum of squares [units * kSlabLanes], or null
    float *norm;             // per-row ||x||^2 of the owner rows, or null
    float lam, lr, xi;
    int32_t clip, degree;
    int32_t *err;
    int32_t epoch;
    int32_t skip_after_nonfinite;
};

// fp32 factors with k in {8, 16, 32, 64}.
bool slab_supported(int K, int prec);
int slab_rows(int K);  // C for rank K
void launch_slab_seg(const int2 *stream, const int64_t *ptr, int32_t rows, int32_t n_slabs, int32_t C,
                     uint32_t *seg, hipStream_t s);
// The slab pass's copy of a stream (see SlabArgs): run (x, s) of the
// bucketed stream, cells seg[s * rows + x] .. seg[(s + 1) * rows + x] - 1,
// goes to records pseg[s * rows + x] .. pseg[s * rows + x + 1] - 1, the
// cells whose other index has parity (x >> 3) & 1 first (see slab.hip),
// then pads.
void launch_slab_order(const int2 *stream, const uint32_t *seg, int32_t rows, int32_t n_slabs, int32_t C,
                       const uint32_t *pseg, uint4 *sblk, hipStream_t s);
// The pass over n_units workgroups.  With U == 1 it updates the rows itself;
// with U > 1 (and not loss-only) launch_slab_finish then adds each row's U
// partial sums and updates it.
void launch_slab_pass(int K, bool loss_only, const SlabArgs &a, int64_t n_units, hipStream_t s,
                      hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
void launch_slab_finish(int K, const SlabArgs &a, hipStream_t s, hipEvent_t ev0 = nullptr,
                        hipEvent_t ev1 = nullptr);
// The P pass (a0, n0 workgroups) and the Q pass (a1, n1) of one simultaneous
// step in one launch (one slab size on both sides), and both finishes
// (both sides with U > 1) in one launch.
void launch_slab_pass_pair(int K, const SlabArgs &a0, int64_t n0, const SlabArgs &a1, int64_t n1, hipStream_t s,
                           hipEvent_t ev0 = nullptr, hipEvent_t ev1 = nullptr);
void launch_slab_finish_pair(int K, const SlabArgs &a0, const SlabArgs &a1, hipStream_t s, hipEvent_t ev0 = nullptr,
                             hipEvent_t ev1 = nullptr);

// ------------------------------------------------- exact extension solve
struct RidgeArgs {
    const int2 *stream;   // chunk cells bucketed by free row: {fixed id, value bits}
    const int64_t *ptr;   // bucket pointers [rows + 1]
    int64_t rows;         // free rows
    const float *F;       // fixed factors (rows indexed by fixed id), fp32
    float lambda;
    float *X;             // rows x K results
    int32_t *err;
    // Gradient steps in Gram form (launch_extend_gram): the free rows with at
    // least gram_min cells take `steps` steps of Eq. 5 (lr, the step option
    // `degree`, the clip and xi as in the template fit) from x = 0.
    int64_t gram_min;
    int32_t steps, clip, degree;
    float lr, xi;
};
bool ridge_supported(int K);
void launch_ridge_rows(int K, const RidgeArgs &a, hipStream_t s);
// The smallest free-row length for which the Gram form of `steps` gradient
// steps is cheaper than the per-cell form at rank K with n_fixed fixed rows
// (0: never).
int64_t extend_gram_min(int K, int32_t steps, int32_t clip, int64_t n_fixed);
void launch_extend_gram(int K, const RidgeArgs &a, hipStream_t s);

// ---------------------------------------- extension by Adam on coefficients
struct AdamArgs {
    const int2 *stream;   // chunk cells bucketed by free line: {fixed id, value bits}
    const int64_t *ptr;   // bucket pointers [n_free + 1]
    int64_t n_free;
    const float *F;       // fixed factors (rows indexed by fixed id), fp32, K per row
    const float *B;       // basis factors, n_b x K, fp32
    int64_t n_b;
    int32_t n_slices;     // ceil(n_b / 256)
    float *C, *M, *V;     // coefficients and moments, n_free x n_b
    float *qpart;         // partial products B^T c_f per slice, n_free x n_slices x K
    float *gt;            // dL/dx_f, n_free x K
    float *X;             // results B^T c_f, n_free x K
    float lambda, lr, beta1, beta2, eps;
    int32_t *err;
    int32_t skip_after_nonfinite;
    // the item pass that forms each step's gradient: device work plan over
    // the chunk's buckets (item_off: n_free + 1, items), a bound on its item
    // count, its item length, its split-bucket sums (n_items_ub x K) and the
    // rows of F
    const uint32_t *item_off;
    const int32_t *items;
    int64_t n_items_ub;
    int32_t E;
    float *carry;
    int64_t n_fixed;
};
bool adam_supported(int K);
int32_t adam_slices(int64_t n_b);
void launch_adam(int K, const AdamArgs &a, int32_t steps, hipStream_t s);

// ----------------------------------------------------------- dense tiles
struct DenseArgs {
    const uint16_t *X;        // owner side bf16 copy (rows x K)
    const uint16_t *Y;        // other side bf16 copy (y_rows x K)
    int64_t rows, y_rows;
    // Work: segments of at most a few dozen consecutive dense tiles of one
    // stripe (16 owner rows), one wave each.
    int64_t n_segs;
    const int32_t *seg_order;   // the segment the w-th wave of the launch takes
    const uint32_t *seg_tile;   // tiles of segment g: seg_tile[g] .. seg_tile[g + 1]
    const int32_t *seg_stripe;  // stripe of segment g
    const uint32_t *stripe_seg; // segments of stripe s: stripe_seg[s] .. stripe_seg[s + 1]
    const int32_t *tile_other;  // other-side tile index (t0 / 16) of each dense tile
    const float *R;             // dense tiles, owner-major 16 x 16 fp32, NaN = not observed
    float *gd;                  // rows x K: gradient sums of the dense cells (stripes with tiles)
    float *part;                // n_segs x 16 x K: partial sums of segments of split stripes
    const int32_t *multi;       // stripes with more than one segment
    int64_t n_multi;
    float *e2;                  // per segment residual sum of squares, or null
    int32_t *err;
    int32_t epoch;
    int32_t skip_after_nonfinite;
};

// bf16 factors with k in {16, 32, 64, 128}.
bool dense_supported(int K, int prec);
// The tile kernel, then (when a stripe has several segments) the kernel that
// adds their partial sums in segment order; ev0 / ev1 bracket both.
// Both sides' tile passes (and combines) of one simultaneous step in one
// launch each (full-gradient, not loss-only).
void launch_dense_pass_pair(int K, const DenseArgs &a0, const DenseArgs &a1, hipStream_t s, hipEvent_t ev0 = nullptr,
                            hipEvent_t ev1 = nullptr);
void launch_dense_pass(int K, bool loss_only, const DenseArgs &a, hipStream_t s, hipEvent_t ev0 = nullptr,
                       hipEvent_t ev1 = nullptr);
// Build steps (see dense.hip).  Tiles: t = ti * n_tj + tj over 16 x 16 blocks.
void tile_count(const int2 *stream, const int64_t *ptr, int32_t rows, int64_t n_tj, uint32_t *cnt, hipStream_t s);
void tile_flag(const uint32_t *cnt, int64_t n_ti, int64_t n_tj, uint32_t thr, bool transpose, uint32_t *flag,
               hipStream_t s);
void tile_list(const uint32_t *flag, const uint32_t *idx, int64_t n_stripes, int64_t n_other, int32_t *tile_other,
               uint32_t *tile_ptr, hipStream_t s);
void sparse_count(const int2 *stream, const int64_t *ptr, int32_t rows, int side, int64_t n_tj,
                  const uint32_t *flag_p, int64_t *count, hipStream_t s);
void tile_split(const int2 *stream, const int64_t *ptr, int32_t rows, int side, int64_t n_ti, int64_t n_tj,
                const uint32_t *flag_p, const uint32_t *idx_p, const uint32_t *flag_q, const uint32_t *idx_q,
                float *Rp, float *Rq, const int64_t *sparse_ptr, int2 *sparse, hipStream_t s);
void fill_nan(float *p, int64_t n, hipStream_t s);

}  // namespace tsid
