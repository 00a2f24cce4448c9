// Dense head tiles of the template fit on MFMA (Section 5.1, Tensor-Core
// batching).  A most-observed (Zipf) template concentrates its cells in its
// head: a third to two thirds of them lie in 16 x 16 tiles that are at
// least 15% full.  For those tiles the residuals and both gradients of Eqs. 3-4
// are dense 16 x 16 x k products, so they run as bf16 MFMA with fp32
// accumulation instead of one cell at a time; the remaining cells stay on the
// item pass, which adds each row's dense gradient sum before the update of
// Eq. 5.
//
// Orientation: a pass has an owner side (the factor it updates: P in the P
// pass, Q in the Q pass) and an other side.  A dense tile covers owner rows
// o0 .. o0+15 and other rows t0 .. t0+15; its observed values are stored
// owner-major (16 x 16 fp32, NaN where a cell is not observed).
//
// Work: a stripe (16 owner rows) and its dense tiles in order of t0.  A Zipf
// head stripe meets nearly every block of the other side, so a stripe's tile
// list is cut into segments of a few dozen tiles, one wave each; a stripe of
// one segment writes its gradient sums directly, the segments of a longer
// one write partial sums that k_dense_combine adds in segment order.  Per
// tile (v_mfma_f32_16x16x32_bf16):
//  1. S^T = Y_t X_t^T (other x owner), k/32 MFMAs over the bf16 copies.  The
//     result lane l holds is S[owner l%16][other 4(l/16)+j]: the A-operand
//     rows of E in step 3, so no shuffle is needed.
//  2. E = R - S on observed cells, 0 elsewhere; E^2 feeds the loss.
//  3. G_X += E Y_t, one k = 32 MFMA per 16 coordinates: E enters as a bf16
//     high part and a bf16 remainder stacked along k (about 16 mantissa
//     bits of the fp32 residual), the B operand Y_t[other][coordinate]
//     comes from an LDS copy of the tile's other rows; the bf16 factor
//     values are exact.
// A wave keeps two tiles' loads in flight.  No atomics: every sum is taken
// in a fixed order, so results repeat bit for bit.
#include <hip/hip_ext.h>

#include "internal.h"

namespace tsid {

namespace {

#ifndef TSID_DENSE_WAVES
#define TSID_DENSE_WAVES 4
#endif
constexpr int kDenseWaves = TSID_DENSE_WAVES;  // waves (segments) per workgroup

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
typedef float fl2 __attribute__((ext_vector_type(2)));
typedef short s4 __attribute__((ext_vector_type(4)));

// Shapes for rank K: 32-coordinate chunks (the k-steps of step 1), 16-
// coordinate blocks (the gradient products of step 3) and the row stride of
// the LDS copy of a tile's other rows (bf16; 16 bytes of padding put the
// 16-byte row writes of 16 lanes and the 2-byte column reads of 64 lanes on
// distinct banks).
template <int K>
struct DenseShape {
    static constexpr int NC = (K + 31) / 32;
    static constexpr int NB = K / 16;
    static constexpr int ROW = K + 8;
};

// Eight bf16 (16 bytes) of row `row` of a bf16 factor table from coordinate
// c0; zeros for c0 >= K (rank 16 fills half of a 32-coordinate chunk).
template <int K>
__device__ __forceinline__ bf8 load8_bf16(const uint16_t *X, int64_t row, int c0) {
    const int c = (K % 32 == 0 || c0 < K) ? c0 : K - 8;
    uint4 w = *reinterpret_cast<const uint4 *>(X + row * K + c);
    if (K % 32 != 0 && c0 >= K) w = make_uint4(0u, 0u, 0u, 0u);
    return __builtin_bit_cast(bf8, w);
}

// Two fp32 to two bf16 (round to nearest even, v_cvt_pk_bf16_f32), packed.
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((fl2){a, b}, bf2));
}

// A tile's operands: its 16 other rows t0 .. t0 + 15 read as whole rows
// (lane l of load c holds the 16 bytes at chunk l % (k/8) of row
// (64 c + l) / (k/8); whole 128-byte lines per load instead of a quarter of
// 16 lines, which halves the L1 tag work per tile) and the tile values
// (owner lr, others 4 lq .. 4 lq + 3).
template <int K>
__device__ __forceinline__ void load_tile(const DenseArgs &A, int32_t other, uint32_t t, int lr, int lq,
                                          bf8 (&y)[DenseShape<K>::NC], float4 &r) {
    constexpr int LPR = K / 8;  // lanes per row
    const int64_t t0 = (int64_t)other * 16;
    const int lane = lq * 16 + lr;
#pragma unroll
    for (int c = 0; c < DenseShape<K>::NC; ++c) {
        const int rr = (c * 64 + lane) / LPR;  // row of the tile (16 and up only at k = 16: not used)
        const int64_t row = t0 + (rr < 16 ? rr : 15);
        // rows past the table repeat its last row (their cells are all unobserved)
        const int64_t yrow = row < A.y_rows ? row : A.y_rows - 1;
        y[c] = __builtin_bit_cast(bf8, *reinterpret_cast<const uint4 *>(A.Y + yrow * K + (lane % LPR) * 8));
    }
    r = *reinterpret_cast<const float4 *>(A.R + (int64_t)t * 256 + lr * 16 + 4 * lq);
}

// Steps 1-3 for one tile (v_mfma_f32_16x16x32_bf16: lane l holds
// A[l%16][8(l/16)+j], B[8(l/16)+j][l%16], j = 0..7, and C[4(l/16)+j][l%16],
// j = 0..3): e^2 into e2, E Y_t into acc.  yl: this wave's LDS copy of the
// tile's other rows, through which the whole-row loads reach both MFMA
// layouts.  valid = false (a stand-in past the end of the segment) zeroes
// the residuals, so the tile adds exactly nothing.
template <int K, bool LOSS_ONLY>
__device__ __forceinline__ void dense_tile(const bf8 (&yraw)[DenseShape<K>::NC], const float4 &r,
                                           const bf8 (&xb)[DenseShape<K>::NC], f4 (&acc)[DenseShape<K>::NB],
                                           float &e2, uint16_t *yl, int lr, int lq, bool valid) {
    using D = DenseShape<K>;
    constexpr int LPR = K / 8;
    const int lane = lq * 16 + lr;
#pragma unroll
    for (int c = 0; c < D::NC; ++c) {
        const int rr = (c * 64 + lane) / LPR;
        if (rr < 16) *reinterpret_cast<uint4 *>(yl + rr * D::ROW + (lane % LPR) * 8) = __builtin_bit_cast(uint4, yraw[c]);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // the A operand of step 1: row lr, coordinates 32 c + 8 lq .. + 7
    bf8 ya[D::NC];
#pragma unroll
    for (int c = 0; c < D::NC; ++c) {
        uint4 w = make_uint4(0u, 0u, 0u, 0u);
        if (K % 32 == 0 || 8 * lq < K) w = *reinterpret_cast<const uint4 *>(yl + lr * D::ROW + c * 32 + 8 * lq);
        ya[c] = __builtin_bit_cast(bf8, w);
    }
    // 1. S^T = Y_t X_t^T: lane holds S[owner lr][other 4 lq + j]
    f4 st = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < D::NC; ++c) st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ya[c], xb[c], st, 0, 0, 0);
    // 2. residuals of the observed cells
    const float rv[4] = {r.x, r.y, r.z, r.w};
    float e[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        e[j] = (valid && rv[j] == rv[j]) ? rv[j] - st[j] : 0.f;  // NaN marks an unobserved cell
        e2 += e[j] * e[j];
    }
    if constexpr (!LOSS_ONLY) {
        // 3. G += E Y_t with one k = 32 product per 16-coordinate block: the
        // A operand holds the residuals' bf16 high parts in slots 0-3 and
        // their remainders in slots 4-7, the B operand the same four other
        // rows twice (a column of the LDS copy), so the product adds
        // (high + low) Y, about 16 bits of each residual.
        const uint32_t h0 = pk_bf16(e[0], e[1]), h1 = pk_bf16(e[2], e[3]);
        const uint32_t l0 = pk_bf16(e[0] - __uint_as_float(h0 << 16), e[1] - __uint_as_float(h0 & 0xffff0000u));
        const uint32_t l1 = pk_bf16(e[2] - __uint_as_float(h1 << 16), e[3] - __uint_as_float(h1 & 0xffff0000u));
        const bf8 ea = __builtin_bit_cast(bf8, make_uint4(h0, h1, l0, l1));
#pragma unroll
        for (int nb = 0; nb < D::NB; ++nb) {
            // column 16 nb + lr of rows 4 lq .. 4 lq + 3 by one transposing LDS
            // read (ds_read_b64_tr_b16): in each group of 16 lanes, lane i
            // receives element i % 4 of the 8-byte pieces of lanes i / 4,
            // 4 + i / 4, 8 + i / 4 and 12 + i / 4, so lane j of the group
            // points at row 4 lq + j / 4, coordinates 16 nb + 4 (j % 4) .. + 3
            const uint16_t *src = yl + (4 * lq + (lr >> 2)) * D::ROW + nb * 16 + 4 * (lr & 3);
            const uint2 w = __builtin_bit_cast(
                uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                           (__attribute__((address_space(3))) s4 *)(src)));
            const bf8 b = __builtin_bit_cast(bf8, make_uint4(w.x, w.y, w.x, w.y));
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ea, b, acc[nb], 0, 0, 0);
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();  // the tile's reads are done before the next writes
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Waves per SIMD the register allocation aims for (0: the compiler's choice).
#ifndef TSID_DENSE_WPE
#define TSID_DENSE_WPE 0
#endif
#if TSID_DENSE_WPE > 0
#define TSID_DENSE_OCC __attribute__((amdgpu_waves_per_eu(TSID_DENSE_WPE)))
#else
#define TSID_DENSE_OCC
#endif

// Workgroup `bid` of one side's tile pass.
template <int K, bool LOSS_ONLY>
__device__ __forceinline__ void dense_pass_group(const DenseArgs &A, const int64_t bid) {
    using D = DenseShape<K>;
    static_assert(K % 16 == 0, "dense tiles need k a multiple of 16");
    if (A.skip_after_nonfinite) {
        const int32_t f = A.err[ERR_NONFINITE];
        if (f != 0 && f - 1 < A.epoch) return;
    }
    __shared__ uint16_t ylds[kDenseWaves][16 * D::ROW];
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int64_t w = bid * kDenseWaves + wv;
    if (w >= A.n_segs) return;  // whole waves leave together
    const int64_t g = A.seg_order[w];  // segment
    const uint32_t t_beg = A.seg_tile[g], t_end = A.seg_tile[g + 1];  // at least one tile
    const uint32_t last = t_end - 1;
    const int64_t s = A.seg_stripe[g], o0 = s * 16;
    const int lr = lane & 15, lq = lane >> 4;  // row within the tile, quarter
    // other-side indices of a window of 64 tiles, one per lane, so that a
    // tile's loads need no dependent load of its index
    uint32_t wbase = t_beg;
    int32_t win = t_beg + lane < t_end ? A.tile_other[t_beg + lane] : 0;
    // owner rows (B operand of step 1), loaded once per segment
    const int64_t orow = o0 + lr < A.rows ? o0 + lr : A.rows - 1;
    bf8 xb[D::NC];
#pragma unroll
    for (int c = 0; c < D::NC; ++c) xb[c] = load8_bf16<K>(A.X, orow, c * 32 + 8 * lq);
    f4 acc[D::NB];
#pragma unroll
    for (int nb = 0; nb < D::NB; ++nb) acc[nb] = f4{0.f, 0.f, 0.f, 0.f};
    float e2 = 0.f;
    // two tiles in flight: buffer a holds tile t, b tile t + 1 (a segment's
    // last tile stands in for tiles past its end)
    bf8 ya[D::NC], yb[D::NC];
    float4 ra, rb;
    load_tile<K>(A, __builtin_amdgcn_readlane(win, 0), t_beg, lr, lq, ya, ra);
    {
        const uint32_t t1 = t_beg + 1 < t_end ? t_beg + 1 : last;
        load_tile<K>(A, __builtin_amdgcn_readlane(win, (int)(t1 - wbase)), t1, lr, lq, yb, rb);
    }
    for (uint32_t t = t_beg; t < t_end; t += 2) {
        dense_tile<K, LOSS_ONLY>(ya, ra, xb, acc, e2, ylds[wv], lr, lq, true);
        const uint32_t n0 = t + 2 < t_end ? t + 2 : last, n1 = t + 3 < t_end ? t + 3 : last;
        if (n1 - wbase >= 64) {  // next window (n1 - n0 <= 1)
            wbase = n0;
            win = n0 + lane < t_end ? A.tile_other[n0 + lane] : 0;
            // wait for the window here, once per 64 tiles: without a use in
            // this branch the wait would be placed after it, in every
            // iteration, and would drain the other tile's loads as well
            asm volatile("" ::"v"(win));
        }
        load_tile<K>(A, __builtin_amdgcn_readlane(win, (int)(n0 - wbase)), n0, lr, lq, ya, ra);
        dense_tile<K, LOSS_ONLY>(yb, rb, xb, acc, e2, ylds[wv], lr, lq, t + 1 < t_end);
        load_tile<K>(A, __builtin_amdgcn_readlane(win, (int)(n1 - wbase)), n1, lr, lq, yb, rb);
    }
    if constexpr (!LOSS_ONLY) {
        // lane holds G[owner 4 lq + j][coordinate 16 nb + lr]; a stripe with
        // one segment writes its rows' sums, the segments of a split stripe
        // write partial sums that k_dense_combine adds in segment order
        const bool whole = A.stripe_seg[s + 1] - A.stripe_seg[s] == 1;
        float *dst = whole ? A.gd + o0 * K : A.part + g * 16 * K;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (o0 + 4 * lq + j < A.rows) {
#pragma unroll
                for (int nb = 0; nb < D::NB; ++nb) dst[(4 * lq + j) * K + nb * 16 + lr] = acc[nb][j];
            }
        }
    }
    if (A.e2) {
        // fixed-order butterfly over the wave
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) e2 += __shfl_xor(e2, off, 64);
        if (lane == 0) A.e2[g] = e2;
    }
}

template <int K, bool LOSS_ONLY>
__global__ __launch_bounds__(64 * kDenseWaves) TSID_DENSE_OCC void k_dense_pass(const DenseArgs A) {
    dense_pass_group<K, LOSS_ONLY>(A, blockIdx.x);
}

// Both sides' tile passes in one launch (they read only the old factors and
// write disjoint sums): the b0 workgroups of the P side (A0), then the Q
// side's (A1).
template <int K>
__global__ __launch_bounds__(64 * kDenseWaves) TSID_DENSE_OCC void k_dense_pass_pair(const DenseArgs A0,
                                                                                    const DenseArgs A1,
                                                                                    const int32_t b0) {
    const int b = blockIdx.x;
    if (b < b0)
        dense_pass_group<K, false>(A0, b);
    else
        dense_pass_group<K, false>(A1, b - b0);
}

// Gradient sums of the stripes split into several segments: the segments'
// partial sums added in segment order (one workgroup per such stripe, one
// lane per 4 coordinates of a row).
template <int K>
__device__ __forceinline__ void dense_combine_group(const DenseArgs &A, const int64_t bid) {
    if (A.skip_after_nonfinite) {
        const int32_t f = A.err[ERR_NONFINITE];
        if (f != 0 && f - 1 < A.epoch) return;
    }
    const int64_t s = A.multi[bid], o0 = s * 16;
    const uint32_t g0 = A.stripe_seg[s], g1 = A.stripe_seg[s + 1];
    for (int idx = threadIdx.x; idx < 16 * K / 4; idx += 256) {
        const int row = idx / (K / 4), c = (idx % (K / 4)) * 4;
        if (o0 + row >= A.rows) break;  // rows past the table (idx grows with row)
        const float *p = A.part + row * K + c;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        uint32_t g = g0;
        for (; g + 4 <= g1; g += 4) {
            float4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const float4 *>(p + (int64_t)(g + u) * 16 * K);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                acc.x += v[u].x;
                acc.y += v[u].y;
                acc.z += v[u].z;
                acc.w += v[u].w;
            }
        }
        for (; g < g1; ++g) {
            const float4 v = *reinterpret_cast<const float4 *>(p + (int64_t)g * 16 * K);
            acc.x += v.x;
            acc.y += v.y;
            acc.z += v.z;
            acc.w += v.w;
        }
        *reinterpret_cast<float4 *>(A.gd + (o0 + row) * K + c) = acc;
    }
}

template <int K>
__global__ __launch_bounds__(256) void k_dense_combine(const DenseArgs A) {
    dense_combine_group<K>(A, blockIdx.x);
}

// Both sides' combines in one launch (the P side's b0 stripes first).
template <int K>
__global__ __launch_bounds__(256) void k_dense_combine_pair(const DenseArgs A0, const DenseArgs A1, const int32_t b0) {
    const int b = blockIdx.x;
    if (b < b0)
        dense_combine_group<K>(A0, b);
    else
        dense_combine_group<K>(A1, b - b0);
}

// ---------------------------------------------------------------- build
// Cells per 16 x 16 tile (a build-time histogram).
__global__ void k_tile_count(const int2 *stream, const int64_t *ptr, int32_t rows, int64_t n_tj,
                             uint32_t *cnt) {
    const int64_t x = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
    if (x >= rows) return;
    const int lane = threadIdx.x & 63;
    for (int64_t j = ptr[x] + lane; j < ptr[x + 1]; j += 64)
        atomicAdd(cnt + (x >> 4) * n_tj + (stream[j].x >> 4), 1u);
}

// flag[t] = 1 if tile t (row-major: t = ti * n_tj + tj; with transpose, the
// flag of column-major position t' = tj * n_ti + ti) holds at least `thr`
// cells.
__global__ void k_tile_flag(const uint32_t *cnt, int64_t n_ti, int64_t n_tj, uint32_t thr, int transpose,
                            uint32_t *flag) {
    const int64_t n = n_ti * n_tj;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
        const int64_t src = transpose ? (t % n_ti) * n_tj + t / n_ti : t;
        flag[t] = cnt[src] >= thr ? 1u : 0u;
    }
}

// After exclusive scans of the flags: the other-side tile index of each dense
// tile, in owner-stripe order, and the stripe pointers.
__global__ void k_tile_list(const uint32_t *flag, const uint32_t *idx, int64_t n_stripes, int64_t n_other,
                            int32_t *tile_other, uint32_t *tile_ptr) {
    const int64_t n = n_stripes * n_other;
    for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += (int64_t)gridDim.x * blockDim.x) {
        if (flag[t]) tile_other[idx[t]] = (int32_t)(t % n_other);
        if (t % n_other == 0) tile_ptr[t / n_other] = idx[t];
    }
}

// Values of the dense cells into their tiles, both orientations; the other
// cells of the buckets are appended (in order) to the sparse streams, whose
// bucket counts come from k_sparse_count.  One wave per bucket of the CSR
// (rows) or the CSC (columns); `side` says which.
__global__ void k_tile_split(const int2 *stream, const int64_t *ptr, int32_t rows, int side, int64_t n_ti,
                             int64_t n_tj, const uint32_t *flag_p, const uint32_t *idx_p,
                             const uint32_t *flag_q, const uint32_t *idx_q, float *Rp, float *Rq,
                             const int64_t *sparse_ptr, int2 *sparse) {
    const int64_t x = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
    if (x >= rows) return;
    const int lane = threadIdx.x & 63;
    int64_t out = sparse_ptr[x];
    for (int64_t j0 = ptr[x]; j0 < ptr[x + 1]; j0 += 64) {
        const int64_t j = j0 + lane;
        const bool in = j < ptr[x + 1];
        int2 c = make_int2(0, 0);
        bool dense = false;
        if (in) {
            c = stream[j];
            const int64_t a = side ? c.x : x, b = side ? x : c.x;  // template row, column
            const int64_t tp = (a >> 4) * n_tj + (b >> 4), tq = (b >> 4) * n_ti + (a >> 4);
            dense = flag_p[tp] != 0;
            if (dense && side == 0) {  // each cell once: from the CSR
                Rp[(int64_t)idx_p[tp] * 256 + (a & 15) * 16 + (b & 15)] = __int_as_float(c.y);
                Rq[(int64_t)idx_q[tq] * 256 + (b & 15) * 16 + (a & 15)] = __int_as_float(c.y);
            }
        }
        const bool keep = in && !dense;
        const uint64_t m = __ballot(keep);
        const uint32_t before = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        if (keep) sparse[out + before] = c;
        out += __popcll(m);
    }
}

// Cells of each bucket outside dense tiles.
__global__ void k_sparse_count(const int2 *stream, const int64_t *ptr, int32_t rows, int side, int64_t n_tj,
                               const uint32_t *flag_p, int64_t *count) {
    const int64_t x = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
    if (x >= rows) return;
    const int lane = threadIdx.x & 63;
    int64_t c = 0;
    for (int64_t j = ptr[x] + lane; j < ptr[x + 1]; j += 64) {
        const int64_t o = stream[j].x;
        const int64_t a = side ? o : x, b = side ? x : o;
        c += flag_p[(a >> 4) * n_tj + (b >> 4)] == 0;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
    if (lane == 0) count[x] = c;
}

__global__ void k_fill_nan(float *p, int64_t n) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x)
        p[j] = __int_as_float(0x7fc00000);
}

int grid_of(int64_t n, int per_block) {
    int64_t g = (n + per_block - 1) / per_block;
    if (g < 1) g = 1;
    return (int)(g > 65536 * 4 ? 65536 * 4 : g);
}

template <int K>
void dense_pass_k(bool loss_only, const DenseArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    const unsigned grid = (unsigned)((a.n_segs + kDenseWaves - 1) / kDenseWaves);
    const bool combine = !loss_only && a.n_multi > 0;
    if (loss_only)
        hipExtLaunchKernelGGL(k_dense_pass<K, true>, dim3(grid), dim3(64 * kDenseWaves), 0, s, ev0, ev1, 0, a);
    else
        hipExtLaunchKernelGGL(k_dense_pass<K, false>, dim3(grid), dim3(64 * kDenseWaves), 0, s, ev0,
                              combine ? nullptr : ev1, 0, a);
    TSID_HIP(hipGetLastError());
    if (combine) {
        hipExtLaunchKernelGGL(k_dense_combine<K>, dim3((unsigned)a.n_multi), dim3(256), 0, s, nullptr, ev1, 0, a);
        TSID_HIP(hipGetLastError());
    }
}

// Both sides' tile passes, then both combines (ev0 at the first launch's
// start, ev1 at the last one's end); a side without segments runs alone.
template <int K>
void dense_pass_pair_k(const DenseArgs &a0, const DenseArgs &a1, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (a0.n_segs <= 0 || a1.n_segs <= 0) {
        if (a0.n_segs > 0) dense_pass_k<K>(false, a0, s, ev0, ev1);
        if (a1.n_segs > 0) dense_pass_k<K>(false, a1, s, ev0, ev1);
        return;
    }
    const int64_t g0 = (a0.n_segs + kDenseWaves - 1) / kDenseWaves, g1 = (a1.n_segs + kDenseWaves - 1) / kDenseWaves;
    if (g0 + g1 > INT32_MAX || a0.n_multi + a1.n_multi > INT32_MAX) fail(TSID_E_INVAL, "too many tile segments");
    const bool c0 = a0.n_multi > 0, c1 = a1.n_multi > 0;
    hipExtLaunchKernelGGL(k_dense_pass_pair<K>, dim3((unsigned)(g0 + g1)), dim3(64 * kDenseWaves), 0, s, ev0,
                          (c0 || c1) ? nullptr : ev1, 0, a0, a1, (int32_t)g0);
    TSID_HIP(hipGetLastError());
    if (c0 && c1)
        hipExtLaunchKernelGGL(k_dense_combine_pair<K>, dim3((unsigned)(a0.n_multi + a1.n_multi)), dim3(256), 0, s,
                              nullptr, ev1, 0, a0, a1, (int32_t)a0.n_multi);
    else if (c0 || c1)
        hipExtLaunchKernelGGL(k_dense_combine<K>, dim3((unsigned)(c0 ? a0.n_multi : a1.n_multi)), dim3(256), 0, s,
                              nullptr, ev1, 0, c0 ? a0 : a1);
    TSID_HIP(hipGetLastError());
}

}  // namespace

void launch_dense_pass_pair(int K, const DenseArgs &a0, const DenseArgs &a1, hipStream_t s, hipEvent_t ev0,
                            hipEvent_t ev1) {
    switch (K) {
        case 16: dense_pass_pair_k<16>(a0, a1, s, ev0, ev1); break;
        case 32: dense_pass_pair_k<32>(a0, a1, s, ev0, ev1); break;
        case 64: dense_pass_pair_k<64>(a0, a1, s, ev0, ev1); break;
        case 128: dense_pass_pair_k<128>(a0, a1, s, ev0, ev1); break;
        default: fail(TSID_E_INVAL, "dense tiles need k in {16, 32, 64, 128}");
    }
}

bool dense_supported(int K, int prec) { return prec == TSID_BF16 && K >= 16 && K % 16 == 0 && K <= 128; }

void launch_dense_pass(int K, bool loss_only, const DenseArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (a.n_segs <= 0) return;
    switch (K) {
        case 16: dense_pass_k<16>(loss_only, a, s, ev0, ev1); break;
        case 32: dense_pass_k<32>(loss_only, a, s, ev0, ev1); break;
        case 64: dense_pass_k<64>(loss_only, a, s, ev0, ev1); break;
        case 128: dense_pass_k<128>(loss_only, a, s, ev0, ev1); break;
        default: fail(TSID_E_INVAL, "dense tiles need k in {16, 32, 64, 128}");
    }
}

void tile_count(const int2 *stream, const int64_t *ptr, int32_t rows, int64_t n_tj, uint32_t *cnt, hipStream_t s) {
    if (rows <= 0) return;
    k_tile_count<<<(unsigned)((rows + 3) / 4), 256, 0, s>>>(stream, ptr, rows, n_tj, cnt);
    TSID_HIP(hipGetLastError());
}

void tile_flag(const uint32_t *cnt, int64_t n_ti, int64_t n_tj, uint32_t thr, bool transpose, uint32_t *flag,
               hipStream_t s) {
    if (n_ti * n_tj <= 0) return;
    k_tile_flag<<<grid_of(n_ti * n_tj, 256), 256, 0, s>>>(cnt, n_ti, n_tj, thr, transpose ? 1 : 0, flag);
    TSID_HIP(hipGetLastError());
}

void tile_list(const uint32_t *flag, const uint32_t *idx, int64_t n_stripes, int64_t n_other, int32_t *tile_other,
               uint32_t *tile_ptr, hipStream_t s) {
    if (n_stripes * n_other <= 0) return;
    k_tile_list<<<grid_of(n_stripes * n_other, 256), 256, 0, s>>>(flag, idx, n_stripes, n_other, tile_other,
                                                                  tile_ptr);
    TSID_HIP(hipGetLastError());
}

void sparse_count(const int2 *stream, const int64_t *ptr, int32_t rows, int side, int64_t n_tj,
                  const uint32_t *flag_p, int64_t *count, hipStream_t s) {
    if (rows <= 0) return;
    k_sparse_count<<<(unsigned)((rows + 3) / 4), 256, 0, s>>>(stream, ptr, rows, side, n_tj, flag_p, count);
    TSID_HIP(hipGetLastError());
}

void tile_split(const int2 *stream, const int64_t *ptr, int32_t rows, int side, int64_t n_ti, int64_t n_tj,
                const uint32_t *flag_p, const uint32_t *idx_p, const uint32_t *flag_q, const uint32_t *idx_q,
                float *Rp, float *Rq, const int64_t *sparse_ptr, int2 *sparse, hipStream_t s) {
    if (rows <= 0) return;
    k_tile_split<<<(unsigned)((rows + 3) / 4), 256, 0, s>>>(stream, ptr, rows, side, n_ti, n_tj, flag_p, idx_p,
                                                            flag_q, idx_q, Rp, Rq, sparse_ptr, sparse);
    TSID_HIP(hipGetLastError());
}

void fill_nan(float *p, int64_t n, hipStream_t s) {
    if (n <= 0) return;
    k_fill_nan<<<grid_of(n, 256), 256, 0, s>>>(p, n);
    TSID_HIP(hipGetLastError());
}

}  // namespace tsid
