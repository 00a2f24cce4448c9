// Multi-view similarity term of the item update (Section 5.1, with the item
// similarity matrix S of Eq. 1 over the template's columns).  The objective
// gains (beta / 2) sum_(i, i') S_ii' ||q_i - q_i'||^2 for a symmetric S, whose
// gradient with respect to q_i is 2 beta sum_i' S_ii' (q_i - q_i'): the term
// the update adds to the item factors.
//
// One launch per epoch, before the Q pass, reads Q_t (the fp32 master) and
// leaves per column i
//   gs[i] = sum_e S_e (q_i - q_col[e])          (k numbers; the Q pass adds
//                                                2 beta gs[i] to the gradient)
//   se[i] = sum_e S_e ||q_i - q_col[e]||^2      (the loss term, summed with
//                                                weight beta / 2)
// over the entries e of row i of S.  One wave per column, lanes over the
// coordinates (two per lane at k = 128); each neighbour row is one coalesced
// read.  The sums run in entry order and the lanes' squared norms are added
// by a fixed butterfly, so the result repeats bit for bit.
#include "internal.h"

namespace tsid {

namespace {

constexpr int kSimWaves = 4;

template <int K>
__global__ __launch_bounds__(64 * kSimWaves) void k_sim_terms(const int64_t *ptr, const int32_t *col,
                                                               const float *val, int32_t n, const float *Q,
                                                               float *gs, float *se) {
    constexpr int CPL = (K + 63) / 64;  // coordinates per lane
    const int64_t i = (int64_t)blockIdx.x * kSimWaves + (threadIdx.x >> 6);
    if (i >= n) return;  // whole waves leave together
    const int lane = threadIdx.x & 63;
    float qi[CPL], g[CPL];
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        const int c = lane + 64 * j;
        qi[j] = c < K ? Q[i * K + c] : 0.f;
        g[j] = 0.f;
    }
    float d2 = 0.f;
    const int64_t e1 = ptr[i + 1];
    for (int64_t e = ptr[i]; e < e1; ++e) {
        const int64_t r = col[e];
        const float w = val[e];
        float part = 0.f;
#pragma unroll
        for (int j = 0; j < CPL; ++j) {
            const int c = lane + 64 * j;
            if (c < K) {
                const float d = qi[j] - Q[r * K + c];
                g[j] = fmaf(w, d, g[j]);
                part = fmaf(d, d, part);
            }
        }
        d2 = fmaf(w, part, d2);
    }
#pragma unroll
    for (int j = 0; j < CPL; ++j) {
        const int c = lane + 64 * j;
        if (c < K) gs[i * K + c] = g[j];
    }
    if (se) {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) d2 += __shfl_xor(d2, off, 64);
        if (lane == 0) se[i] = d2;
    }
}

template <int K>
void sim_k(const int64_t *ptr, const int32_t *col, const float *val, int32_t n, const float *Q, float *gs,
           float *se, hipStream_t s) {
    hipLaunchKernelGGL(k_sim_terms<K>, dim3((unsigned)ceil_div(n, kSimWaves)), dim3(64 * kSimWaves), 0, s, ptr,
                       col, val, n, Q, gs, se);
    TSID_HIP(hipGetLastError());
}

}  // namespace

void launch_sim_terms(int K, const int64_t *ptr, const int32_t *col, const float *val, int32_t n, const float *Q,
                      float *gs, float *se, hipStream_t s) {
    if (n <= 0) return;
    switch (K) {
        case 8: sim_k<8>(ptr, col, val, n, Q, gs, se, s); break;
        case 16: sim_k<16>(ptr, col, val, n, Q, gs, se, s); break;
        case 32: sim_k<32>(ptr, col, val, n, Q, gs, se, s); break;
        case 64: sim_k<64>(ptr, col, val, n, Q, gs, se, s); break;
        case 128: sim_k<128>(ptr, col, val, n, Q, gs, se, s); break;
        default: fail(TSID_E_INVAL, "unsupported rank");
    }
}

}  // namespace tsid
