// Exact one-sided solve of an extension chunk (Section 5.2; Eq. 6 in factored
// form): with the fixed side's factors held constant, each free row x_f is
// the ridge regression
//   x_f = argmin sum_(u in cells of f) (r_u - p_u . x)^2 + lambda ||x||^2
//       = (sum_u p_u p_u^T + lambda I)^{-1} sum_u r_u p_u,
// the fixed point that the gradient steps of k_extend_steps approach (the
// alternating-least-squares step of the paper's Stage II).  Everything is
// fp64: the Gram matrix of a row with fewer cells than k is singular up to
// lambda, and fp32 would lose the directions lambda alone fixes.
//
// One wave per free row:
//  1. Gram and right-hand side.  Four cells at a time, each lane loads one
//     coordinate of each 16-coordinate block of one cell's fixed row (lane l:
//     cell l/16, coordinate 16 I + l%16), which is at once the A operand
//     A[l%16][l/16] and the B operand B[l/16][l%16] of v_mfma_f64_16x16x4f64,
//     so block (I, J) of the Gram matrix accumulates with one MFMA per block
//     pair I <= J (10 at k = 64).  Lane l, slot j of a result holds
//     C[4 j + l/16][l%16].  The right-hand side accumulates per lane and is
//     summed over the four cell slots at the end.
//  2. The blocks go through LDS (and their mirror images), lane i reads row i
//     and adds lambda on the diagonal.
//  3. Cholesky G = L L^T, right-looking, with row i of the trailing matrix in
//     lane i's registers: per column j, lane j's diagonal and every lane's
//     L[i][j] are broadcast with readlane, and each lane updates its row.
//     Entries above the diagonal are updated too and never read.
//  4. L z = b column by column in registers, then L^T x = z column by column
//     with the rows of L read back from LDS.
// A pivot that is not positive (lambda = 0 and fewer independent cells than
// k) raises the non-finite error; a row without cells gets x = 0.
#include <hip/hip_ext.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>

#include "internal.h"

namespace tsid {

namespace {

typedef double d4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double readlane_f64(double v, int l) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int K>
struct RidgeShape {
    static constexpr int NB = (K + 15) / 16;          // 16-coordinate blocks
    static constexpr int NP = NB * (NB + 1) / 2;      // block pairs I <= J
    static constexpr int PITCH = K + 1;               // LDS row pitch (doubles)
};

// Gram blocks (block pairs I <= J) and right-hand side of one free row's
// cells b0 .. b1 (b1 > b0), by one wave with the operand layout above.  Four
// groups of four cells are loaded before their products, so each lane keeps
// four gathers per block in flight; loads past the row's end re-read its
// last cell and are masked.
template <int K>
__device__ __forceinline__ void gram_line(const RidgeArgs &A, int64_t b0, int64_t b1, int lane,
                                          d4 (&acc)[RidgeShape<K>::NP], double (&rhs)[RidgeShape<K>::NB]) {
    using S = RidgeShape<K>;
    constexpr int U = 4;
    const int lr = lane & 15, lq = lane >> 4;
#pragma unroll
    for (int q = 0; q < S::NP; ++q) acc[q] = d4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int I = 0; I < S::NB; ++I) rhs[I] = 0.0;
    for (int64_t c0 = b0; c0 < b1; c0 += 4 * U) {
        int2 rec[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t c = c0 + 4 * u + lq;
            rec[u] = A.stream[c < b1 ? c : b1 - 1];
        }
        double pv[U][S::NB], rv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = c0 + 4 * u + lq < b1;
            rv[u] = in ? (double)__int_as_float(rec[u].y) : 0.0;
            const float *p = A.F + (int64_t)rec[u].x * K;
#pragma unroll
            for (int I = 0; I < S::NB; ++I) {
                const int col = (K % 16 == 0 || 16 * I + lr < K) ? 16 * I + lr : K - 1;
                const float v = p[col];
                pv[u][I] = (in && (K % 16 == 0 || 16 * I + lr < K)) ? (double)v : 0.0;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int q = 0;
#pragma unroll
            for (int I = 0; I < S::NB; ++I) {
                rhs[I] = fma(rv[u], pv[u][I], rhs[I]);
#pragma unroll
                for (int J = I; J < S::NB; ++J, ++q)
                    acc[q] = __builtin_amdgcn_mfma_f64_16x16x4f64(pv[u][I], pv[u][J], acc[q], 0, 0, 0);
            }
        }
    }
}

// The Gram blocks and their mirror images to LDS (pitch K + 1); the
// right-hand side summed over the four cell slots, lane i returning b_i.
template <int K>
__device__ __forceinline__ double gram_to_lds(const d4 (&acc)[RidgeShape<K>::NP], double (&rhs)[RidgeShape<K>::NB],
                                              double *G, int lane) {
    using S = RidgeShape<K>;
    const int lr = lane & 15, lq = lane >> 4;
    int q = 0;
#pragma unroll
    for (int I = 0; I < S::NB; ++I) {
#pragma unroll
        for (int J = I; J < S::NB; ++J, ++q) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int row = 16 * I + 4 * j + lq, col = 16 * J + lr;
                if (row < K && col < K) {
                    G[row * S::PITCH + col] = acc[q][j];
                    G[col * S::PITCH + row] = acc[q][j];
                }
            }
        }
    }
    // coordinate i = 16 (i / 16) + i % 16 sits in lane i after the sums
#pragma unroll
    for (int I = 0; I < S::NB; ++I) {
        rhs[I] += __shfl_xor(rhs[I], 16, 64);
        rhs[I] += __shfl_xor(rhs[I], 32, 64);
    }
    double b = 0.0;
#pragma unroll
    for (int I = 0; I < S::NB; ++I) b = (lq == I) ? rhs[I] : b;
    return b;
}

template <int K>
__global__ __launch_bounds__(64) void k_ridge_rows(const RidgeArgs A) {
    using S = RidgeShape<K>;
    __shared__ double G[K * S::PITCH];
    const int lane = threadIdx.x;
    const int64_t f = blockIdx.x;  // free row
    if (f >= A.rows) return;
    const int64_t b0 = A.ptr[f], b1 = A.ptr[f + 1];
    if (b0 == b1) {  // no cells: the minimiser is 0
        if (lane < K) A.X[f * K + lane] = 0.f;
        return;
    }
    // 1.-2. Gram blocks and right-hand side, the blocks through LDS
    d4 acc[S::NP];
    double rhs[S::NB];
    gram_line<K>(A, b0, b1, lane, acc, rhs);
    double b = gram_to_lds<K>(acc, rhs, G, lane);
    __syncthreads();
    const int ri = lane < K ? lane : K - 1;  // lanes past k mirror the last row (never read back)
    double g[K];
#pragma unroll
    for (int c = 0; c < K; ++c) g[c] = G[ri * S::PITCH + c] + ((c == lane) ? (double)A.lambda : 0.0);
    // 3. Cholesky, right-looking; lane i ends with L[i][0..i] in g[0..i]
    bool bad = false;
    double dinv = 1.0;  // 1 / L[i][i] of this lane's row
#pragma unroll
    for (int j = 0; j < K; ++j) {
        const double djj = readlane_f64(g[j], j);
        bad |= !(djj > 0.0);
        const double ljj = sqrt(djj > 0.0 ? djj : 1.0);
        const double inv = 1.0 / ljj;
        const double lij = (lane == j) ? ljj : g[j] * inv;
        dinv = (lane == j) ? inv : dinv;
        g[j] = (lane >= j) ? lij : g[j];
#pragma unroll
        for (int l = j + 1; l < K; ++l) g[l] = fma(-lij, readlane_f64(lij, l), g[l]);
    }
    // 4a. L z = b (column-oriented): lane c finishes z_c, the lanes below take it out
#pragma unroll
    for (int c = 0; c < K; ++c) {
        const double zc = readlane_f64(b * dinv, c);
        b = (lane == c) ? zc : ((lane > c) ? fma(-g[c], zc, b) : b);
    }
    // 4b. L^T x = z: rows of L back through LDS (lane i reads L[r][i])
    __syncthreads();
    if (lane < K) {
#pragma unroll
        for (int c = 0; c < K; ++c)
            if (c <= lane) G[lane * S::PITCH + c] = g[c];
    }
    __syncthreads();
    double x = 0.0;
#pragma unroll
    for (int r = K - 1; r >= 0; --r) {
        const double xr = readlane_f64(b * dinv, r);
        x = (lane == r) ? xr : x;
        if (lane < r) b = fma(-G[r * S::PITCH + lane], xr, b);
    }
    bad = __builtin_amdgcn_ballot_w64(bad) != 0;  // a bad pivot anywhere spoils the whole row
    if (lane < K) {
        const float xf = (float)x;
        A.X[f * K + lane] = xf;
        if (bad || !__builtin_isfinite(xf)) A.err[ERR_NONFINITE] = 1;
    }
}

// One-sided gradient steps in Gram form (Section 5.2's per-row subproblem
// with Eq. 5's update).  With the fixed side held, the gradient of a free
// row's loss is 2 lambda x - 2 (b - G x), G = sum_u p_u p_u^T and
// b = sum_u r_u p_u over the row's cells, so one pass over the cells (fp64,
// as for the exact solve) gives every step: lane i holds row i of G and b_i,
// and a step is the product G x (x broadcast lane by lane), the gradient, the
// step option's scale, the clip and the update, all in fp64 from x = 0.  The
// per-cell kernel (k_extend_steps) gathers every fixed row once per step; for
// rows of at least gram_min cells this one gathers them once.  Rows shorter
// than gram_min are the per-cell kernel's and are left untouched here.
template <int K>
__global__ __launch_bounds__(64) void k_extend_gram(const RidgeArgs A) {
    using S = RidgeShape<K>;
    __shared__ double G[K * S::PITCH];
    const int lane = threadIdx.x;
    const int64_t f = blockIdx.x;
    if (f >= A.rows) return;
    const int64_t b0 = A.ptr[f], b1 = A.ptr[f + 1], deg = b1 - b0;
    if (deg < A.gram_min || deg == 0) return;
    d4 acc[S::NP];
    double rhs[S::NB];
    gram_line<K>(A, b0, b1, lane, acc, rhs);
    const double b = gram_to_lds<K>(acc, rhs, G, lane);
    __syncthreads();
    const int ri = lane < K ? lane : K - 1;  // lanes past k mirror the last row (never stored)
    double g[K];
#pragma unroll
    for (int c = 0; c < K; ++c) g[c] = G[ri * S::PITCH + c];
    const double lam = A.lambda, lr = A.lr, xi = A.xi;
    const double sc = A.degree ? 1.0 / (double)(deg > 1 ? deg : 1) : 1.0;
    double x = 0.0;
    bool bad = false;
    for (int t = 0; t < A.steps; ++t) {
        // G x in four independent sums (a shorter chain of dependent FMAs)
        double gq[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int c = 0; c < K; ++c) gq[c & 3] = fma(g[c], readlane_f64(x, c), gq[c & 3]);
        const double gx = (gq[0] + gq[1]) + (gq[2] + gq[3]);
        const double grad = 2.0 * lam * x - 2.0 * (b - gx);
        double d;
        if (A.clip == 3) {  // the printed asymmetric form: the scale outside the clip
            d = -grad;
            if (d > xi) d = xi;
            d *= sc;
        } else {
            d = -sc * grad;
            if (A.clip && d > xi) d = xi;
        }
        x = fma(lr, d, x);
        bad |= !__builtin_isfinite(x);
    }
    if (lane < K) {
        const float xf = (float)x;
        A.X[f * K + lane] = xf;
        if (bad || !__builtin_isfinite(xf)) A.err[ERR_NONFINITE] = 1;
    }
}

template <int K>
void ridge_k(const RidgeArgs &a, hipStream_t s) {
    hipLaunchKernelGGL(k_ridge_rows<K>, dim3((unsigned)a.rows), dim3(64), 0, s, a);
    TSID_HIP(hipGetLastError());
}

// k = 128: a row of the Gram matrix does not fit one lane's registers, so
// the matrix lives in LDS (128 x 129 doubles, 129 KiB) and a workgroup of
// four waves solves one free row:
//  1. Gram: the 36 block pairs I <= J of the 8 x 8 blocks are dealt to the
//     waves (pair q to wave q % 4); each wave walks all the row's cells, four
//     at a time, with the operand layout of k_ridge_rows, and wave 0 also
//     sums the right-hand side.
//  2. The blocks and their mirror images go to LDS; lambda joins the
//     diagonal.
//  3. Cholesky, right-looking: at column j every thread reads the pivot
//     d = G[j][j], and the trailing lower triangle takes
//     G[r][c] -= G[r][j] G[c][j] / d (two threads per row r > j, alternate
//     columns); column j - 1 is scaled by 1 / sqrt of its pivot in the same
//     phase (no thread reads it any more), so one barrier per column.
//  4. Wave 0 solves L z = b and L^T x = z, lane l holding rows l and l + 64,
//     the pivots of each step broadcast with readlane.
constexpr int kR128 = 128, kR128Pitch = kR128 + 1, kR128Threads = 256;
constexpr int kR128Lds = (kR128 * kR128Pitch + kR128) * 8;

__global__ __launch_bounds__(kR128Threads) void k_ridge_rows_128(const RidgeArgs A) {
    constexpr int K = kR128, NB = K / 16, PITCH = kR128Pitch;
    extern __shared__ double lds[];
    double *G = lds;                  // K x PITCH
    double *rhs = lds + K * PITCH;    // K
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int64_t f = blockIdx.x;
    if (f >= A.rows) return;
    const int lr = lane & 15, lq = lane >> 4;
    const int64_t b0 = A.ptr[f], b1 = A.ptr[f + 1];
    if (b0 == b1) {
        if (tid < K) A.X[f * K + tid] = 0.f;
        return;
    }
    // 1. this wave's block pairs (slot q / 4 of pair q = 4 s + wv)
    d4 acc[9];
#pragma unroll
    for (int q = 0; q < 9; ++q) acc[q] = d4{0.0, 0.0, 0.0, 0.0};
    double rb[NB];
#pragma unroll
    for (int I = 0; I < NB; ++I) rb[I] = 0.0;
    for (int64_t c0 = b0; c0 < b1; c0 += 4) {
        const int64_t c = c0 + lq;
        double pv[NB];
        double rv = 0.0;
#pragma unroll
        for (int I = 0; I < NB; ++I) pv[I] = 0.0;
        if (c < b1) {
            const int2 rec = A.stream[c];
            rv = (double)__int_as_float(rec.y);
            const float *p = A.F + (int64_t)rec.x * K;
#pragma unroll
            for (int I = 0; I < NB; ++I) pv[I] = (double)p[16 * I + lr];
        }
        if (wv == 0) {
#pragma unroll
            for (int I = 0; I < NB; ++I) rb[I] = fma(rv, pv[I], rb[I]);
        }
        int q = 0;
#pragma unroll
        for (int I = 0; I < NB; ++I) {
#pragma unroll
            for (int J = I; J < NB; ++J, ++q)
                if ((q & 3) == wv) acc[q >> 2] = __builtin_amdgcn_mfma_f64_16x16x4f64(pv[I], pv[J], acc[q >> 2], 0, 0, 0);
        }
    }
    // 2. blocks (and mirrors) to LDS; the right-hand side summed over the four cell slots
    {
        int q = 0;
#pragma unroll
        for (int I = 0; I < NB; ++I) {
#pragma unroll
            for (int J = I; J < NB; ++J, ++q) {
                if ((q & 3) != wv) continue;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int row = 16 * I + 4 * j + lq, col = 16 * J + lr;
                    G[row * PITCH + col] = acc[q >> 2][j];
                    G[col * PITCH + row] = acc[q >> 2][j];
                }
            }
        }
    }
    if (wv == 0) {
#pragma unroll
        for (int I = 0; I < NB; ++I) {
            double v = rb[I];
            v += __shfl_xor(v, 16, 64);
            v += __shfl_xor(v, 32, 64);
            if (lq == 0) rhs[16 * I + lr] = v;
        }
    }
    __syncthreads();
    if (tid < K) G[tid * PITCH + tid] += (double)A.lambda;
    __syncthreads();
    // 3. Cholesky
    bool bad = false;
    const int half = tid & 1;
    double dprev = 1.0;  // the previous column's pivot (read before it was overwritten)
    for (int j = 0; j < K; ++j) {
        const double d = G[j * PITCH + j];
        bad |= !(d > 0.0);
        if (j > 0 && tid < K - j + 1) {  // scale column j - 1 (rows j - 1 .. K - 1)
            const int r = j - 1 + tid;
            const double lp = sqrt(dprev > 0.0 ? dprev : 1.0);
            G[r * PITCH + (j - 1)] = r == j - 1 ? lp : G[r * PITCH + (j - 1)] / lp;
        }
        dprev = d;
        const double inv = 1.0 / (d > 0.0 ? d : 1.0);
        const int r = j + 1 + (tid >> 1);
        if (r < K) {
            const double a = G[r * PITCH + j] * inv;
            for (int c = j + 1 + half; c <= r; c += 2) G[r * PITCH + c] = fma(-a, G[c * PITCH + j], G[r * PITCH + c]);
        }
        __syncthreads();
    }
    if (tid == 0)  // the last column's pivot
        G[(K - 1) * PITCH + (K - 1)] = sqrt(dprev > 0.0 ? dprev : 1.0);
    __syncthreads();
    // 4. triangular solves by wave 0: lane l holds rows l and l + 64
    bad = __syncthreads_or(bad);
    if (wv == 0) {
        double bl = rhs[lane], bh = rhs[lane + 64];
        for (int c = 0; c < K; ++c) {  // L z = b, column by column
            const double lcc = G[c * PITCH + c];
            const double zc = (c < 64 ? readlane_f64(bl, c) : readlane_f64(bh, c - 64)) / lcc;
            if (lane == c) bl = zc;
            else if (lane > c) bl = fma(-G[lane * PITCH + c], zc, bl);
            if (lane + 64 == c) bh = zc;
            else if (lane + 64 > c) bh = fma(-G[(lane + 64) * PITCH + c], zc, bh);
        }
        for (int r = K - 1; r >= 0; --r) {  // L^T x = z, row by row
            const double lrr = G[r * PITCH + r];
            const double xr = (r < 64 ? readlane_f64(bl, r) : readlane_f64(bh, r - 64)) / lrr;
            if (lane == r) bl = xr;
            else if (lane < r) bl = fma(-G[r * PITCH + lane], xr, bl);
            if (lane + 64 == r) bh = xr;
            else if (lane + 64 < r) bh = fma(-G[r * PITCH + lane + 64], xr, bh);
        }
        const float xl = (float)bl, xh = (float)bh;
        A.X[f * K + lane] = xl;
        A.X[f * K + lane + 64] = xh;
        if (bad || !__builtin_isfinite(xl) || !__builtin_isfinite(xh)) A.err[ERR_NONFINITE] = 1;
    }
}

void ridge_128(const RidgeArgs &a, hipStream_t s) {
    static const bool lds_ok = [] {
        TSID_HIP(hipFuncSetAttribute(reinterpret_cast<const void *>(k_ridge_rows_128),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, kR128Lds));
        return true;
    }();
    (void)lds_ok;
    hipLaunchKernelGGL(k_ridge_rows_128, dim3((unsigned)a.rows), dim3(kR128Threads), kR128Lds, s, a);
    TSID_HIP(hipGetLastError());
}

}  // namespace

bool ridge_supported(int K) { return K == 8 || K == 16 || K == 32 || K == 64 || K == 128; }

// Where the Gram form pays, per free row of d cells.  Gram form: K^2 r fp64
// multiply-adds per cell on the matrix cores (r: the share of the 16 x 16
// blocks it forms, the pairs I <= J) and, per step, the product G x with x
// broadcast lane by lane (about 3 K wave instructions).  Per-cell form: 2 K
// fp32 multiply-adds per cell and step, and the gathers of the row's fixed
// rows again every step.
//  - A fixed table within one XCD's L2 (4 MiB) serves those gathers from L2,
//    and the forms compare by arithmetic: d = T K / (2 T - K r), when
//    2 T > K r.  Rating-shaped rows (k = 64, 20 steps, a 2 MiB table): all in
//    the per-cell form 16.8 ms, Gram form from 96 / 192 / 384 cells 18.5 /
//    17.3 / 17.2 ms; Scientific rows (k = 32, 2 MiB, about 1,500 cells each)
//    0.112 -> 0.094 s in Gram form.
//  - A larger table is gathered from the memory-side cache or HBM, about
//    4 K / 64 wave instructions' worth per cell and step, and the Gram form
//    pays from d = 192 T / (4 T - K r), when 4 T > K r.  Rating-shaped
//    columns (k = 64, a 123 MB table, about 1,160 cells each): 13.2 -> 7.5 ms
//    (7.49-7.56 ms for thresholds 96 to 384); Scientific columns (k = 32,
//    25.6 MB, about 18,000 cells) 1.38 -> 0.73 s.
// At least 16 cells either way.  Tuning knob TSID_EXT_GRAM_MIN: -1 never,
// n > 0 from n cells on.
int64_t extend_gram_min(int K, int32_t steps, int32_t clip, int64_t n_fixed) {
    if (const char *e = std::getenv("TSID_EXT_GRAM_MIN")) {
        const long long v = std::atoll(e);
        if (v != 0) return v < 0 || K > 64 || clip == 2 || steps < 1 ? 0 : (int64_t)v;
    }
    if (K > 64 || clip == 2 || steps < 1) return 0;
    const int nb = (K + 15) / 16, np = nb * (nb + 1) / 2;
    const double r = (double)np / (double)(nb * nb);
    const bool in_l2 = n_fixed * K * 4 <= (int64_t(4) << 20);
    const double den = (in_l2 ? 2.0 : 4.0) * steps - K * r;
    if (den <= 0.0) return 0;
    const double d = in_l2 ? (double)steps * K / den : 192.0 * steps / den;
    return std::max<int64_t>(16, (int64_t)std::ceil(d));
}

void launch_extend_gram(int K, const RidgeArgs &a, hipStream_t s) {
    if (a.rows <= 0 || a.gram_min <= 0) return;
    if (a.rows > INT32_MAX) fail(TSID_E_INVAL, "too many free rows");
    switch (K) {
        case 8: hipLaunchKernelGGL(k_extend_gram<8>, dim3((unsigned)a.rows), dim3(64), 0, s, a); break;
        case 16: hipLaunchKernelGGL(k_extend_gram<16>, dim3((unsigned)a.rows), dim3(64), 0, s, a); break;
        case 32: hipLaunchKernelGGL(k_extend_gram<32>, dim3((unsigned)a.rows), dim3(64), 0, s, a); break;
        case 64: hipLaunchKernelGGL(k_extend_gram<64>, dim3((unsigned)a.rows), dim3(64), 0, s, a); break;
        default: fail(TSID_E_INVAL, "the Gram-form steps support k in {8, 16, 32, 64}");
    }
    TSID_HIP(hipGetLastError());
}

void launch_ridge_rows(int K, const RidgeArgs &a, hipStream_t s) {
    if (a.rows <= 0) return;
    switch (K) {
        case 8: ridge_k<8>(a, s); break;
        case 16: ridge_k<16>(a, s); break;
        case 32: ridge_k<32>(a, s); break;
        case 64: ridge_k<64>(a, s); break;
        case 128: ridge_128(a, s); break;
        default: fail(TSID_E_INVAL, "the exact extension solve supports k in {8, 16, 32, 64, 128}");
    }
}

}  // namespace tsid
