// Stage II as Eq. 6 states it (Section 5.2): each free line f (a column of
// R outside the template, or a row) is represented in the fixed template
// basis by a coefficient vector c_f with one entry per basis line, and its
// entries are predicted as R*_i c_f.  In factored form R* = P B^T, so the
// prediction of entry (i, f) is p_i . x_f with x_f = B^T c_f (k numbers), and
//   L(C) = sum (r - p . x_f)^2 + lambda ||C||_F^2,
//   dL/dc_f = B g_f + 2 lambda c_f,   g_f = -2 sum (r - p . x_f) p.
// The coefficients move by the Adam method (bias-corrected first and second
// moment estimates, elementwise step lr m^ / (sqrt(w^) + eps)), from C = 0.
//
// A step is four launches, free lines being independent:
//  k_adam_x       x_f from the previous step's partial products (slice order).
//  the item pass  the residual of every entry of f and sum_e e p, with x_f as
//                 the owner row and F the gathered table: the template fit's
//                 per-cell kernel, its sums stored per free line instead of an
//                 update, then k_fixup for the lines split over waves.
//  k_adam_update  one wave per free line and slice of 256 basis lines (four
//                 lanes per basis line, a quarter of its coordinates each):
//                 the gradient of those coefficients, the Adam step, and the
//                 slice's partial product B^T c_f for the next step (the
//                 lanes' terms added in lane order through LDS).
// No atomics: every sum has a fixed order, so results repeat bit for bit.
#include <hip/hip_ext.h>

#include "internal.h"

namespace tsid {

namespace {

constexpr int kAdamUpdWaves = 4;

// x_f = B^T c_f: the slices' partial products of free line f, in slice order.
template <int K>
__global__ __launch_bounds__(256) void k_adam_x(const AdamArgs A) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= A.n_free * K) return;
    const int64_t f = t / K;
    const int c = (int)(t % K);
    float x = 0.f;
    for (int32_t s = 0; s < A.n_slices; ++s) x += A.qpart[(f * A.n_slices + s) * K + c];
    A.X[t] = x;
}

// One wave per free line and slice of 256 basis lines.  Lane l takes basis
// lines l/4 + 16 i of the slice and coordinates 16 (l%4) .. + 15 (K/4 per
// quarter at k < 64): the four lanes of a line read it whole (coalesced) and
// add their partial dot products with two shuffles.
template <int K>
__global__ __launch_bounds__(64 * kAdamUpdWaves) void k_adam_update(const AdamArgs A, float c1, float c2) {
    constexpr int KQ = K / 4;  // coordinates per lane
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int q = lane & 3, rl = lane >> 2;
    const int64_t f = (int64_t)blockIdx.x * kAdamUpdWaves + wv;
    __shared__ float red[kAdamUpdWaves][64][KQ + 1];
    const bool live = f < A.n_free && !(A.skip_after_nonfinite && A.err[ERR_NONFINITE]);
    const int64_t fl = f < A.n_free ? f : A.n_free - 1;
    const int32_t s = blockIdx.y;  // slice of 256 basis lines
    float gv[KQ], qp[KQ];
#pragma unroll
    for (int c = 0; c < KQ; ++c) {
        gv[c] = -2.f * A.gt[fl * K + q * KQ + c];  // dL/dx_f = -2 sum_e e p
        qp[c] = 0.f;
    }
    bool bad = false;
    if (live) {
        for (int i = 0; i < 16; ++i) {
            const int64_t l = (int64_t)s * 256 + i * 16 + rl;
            if (l >= A.n_b) break;  // lines past the basis: the four lanes of a line leave together
            float b[KQ];
            if constexpr (KQ % 4 == 0) {
#pragma unroll
                for (int c = 0; c < KQ; c += 4) {
                    const float4 w = *reinterpret_cast<const float4 *>(A.B + l * K + q * KQ + c);
                    b[c] = w.x;
                    b[c + 1] = w.y;
                    b[c + 2] = w.z;
                    b[c + 3] = w.w;
                }
            } else {
#pragma unroll
                for (int c = 0; c < KQ; ++c) b[c] = A.B[l * K + q * KQ + c];
            }
            float part = 0.f;
#pragma unroll
            for (int c = 0; c < KQ; ++c) part = fmaf(b[c], gv[c], part);
            // the four quarters in a fixed pattern: every lane ends with the same sum
            part += __shfl_xor(part, 1, 64);
            part += __shfl_xor(part, 2, 64);
            const int64_t j = fl * A.n_b + l;
            const float cj = A.C[j];
            const float gr = 2.f * A.lambda * cj + part;
            const float m = A.beta1 * A.M[j] + (1.f - A.beta1) * gr;
            const float w = A.beta2 * A.V[j] + (1.f - A.beta2) * gr * gr;
            const float cn = cj - A.lr * (m * c1) / (sqrtf(w * c2) + A.eps);
            if (q == 0) {
                A.M[j] = m;
                A.V[j] = w;
                A.C[j] = cn;
            }
            bad |= !__builtin_isfinite(cn);
#pragma unroll
            for (int c = 0; c < KQ; ++c) qp[c] = fmaf(b[c], cn, qp[c]);
        }
    }
    // the slice's partial product: the 16 line-lanes of each quarter added in
    // lane order through LDS
#pragma unroll
    for (int c = 0; c < KQ; ++c) red[wv][lane][c] = qp[c];
    __syncthreads();
    if (live) {
        for (int o = lane; o < K; o += 64) {  // coordinate o (two per lane at k = 128)
            const int qq = o / KQ, cc = o % KQ;
            float t = 0.f;
            for (int r = 0; r < 16; ++r) t += red[wv][r * 4 + qq][cc];
            A.qpart[((int64_t)f * A.n_slices + s) * K + o] = t;
        }
    }
    if (bad) A.err[ERR_NONFINITE] = 1;
}

template <int K>
void adam_k(const AdamArgs &a, int32_t steps, hipStream_t st) {
    const double b1 = a.beta1, b2 = a.beta2;
    double b1t = 1.0, b2t = 1.0;
    const dim3 gu((unsigned)((a.n_free + kAdamUpdWaves - 1) / kAdamUpdWaves), (unsigned)a.n_slices);
    const unsigned gx = (unsigned)((a.n_free * K + 255) / 256);
    // the gradient's item pass: owner rows x_f (in X), gathered rows of F,
    // each free line's sum stored in gt instead of an update
    PassArgs g{};
    g.stream = a.stream;
    g.ptr = a.ptr;
    g.items = a.items;
    g.item_off = a.item_off;
    g.item_end = a.item_off + 1;
    g.n_items_dev = a.item_off + a.n_free;
    g.n_items = (int32_t)a.n_items_ub;
    g.rows = (int32_t)a.n_free;
    g.E = a.E;
    g.X = a.X;
    g.Y = a.F;
    g.y_rows = a.n_fixed;
    g.carry = a.carry;
    g.err = a.err;
    g.epoch = INT32_MAX;  // skipped once any step has stored a non-finite flag
    g.skip_after_nonfinite = a.skip_after_nonfinite;
    g.partial_out = a.gt;
    for (int32_t t = 1; t <= steps; ++t) {
        b1t *= b1;
        b2t *= b2;
        hipLaunchKernelGGL(k_adam_x<K>, dim3(gx), dim3(256), 0, st, a);
        TSID_HIP(hipGetLastError());
        launch_item_pass(K, TSID_FP32, false, g, st);
        launch_fixup(K, TSID_FP32, g, st);
        hipLaunchKernelGGL(k_adam_update<K>, gu, dim3(64 * kAdamUpdWaves), 0, st, a, (float)(1.0 / (1.0 - b1t)),
                           (float)(1.0 / (1.0 - b2t)));
        TSID_HIP(hipGetLastError());
    }
    hipLaunchKernelGGL(k_adam_x<K>, dim3(gx), dim3(256), 0, st, a);
    TSID_HIP(hipGetLastError());
}

}  // namespace

bool adam_supported(int K) { return K == 8 || K == 16 || K == 32 || K == 64 || K == 128; }

int32_t adam_slices(int64_t n_b) { return (int32_t)((n_b + 255) / 256); }

void launch_adam(int K, const AdamArgs &a, int32_t steps, hipStream_t s) {
    if (a.n_free <= 0) return;
    switch (K) {
        case 8: adam_k<8>(a, steps, s); break;
        case 16: adam_k<16>(a, steps, s); break;
        case 32: adam_k<32>(a, steps, s); break;
        case 64: adam_k<64>(a, steps, s); break;
        case 128: adam_k<128>(a, steps, s); break;
        default: fail(TSID_E_INVAL, "the Adam extension supports k in {8, 16, 32, 64, 128}");
    }
}

}  // namespace tsid
