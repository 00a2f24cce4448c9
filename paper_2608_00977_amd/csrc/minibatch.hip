// Mini-batch epochs (the in-epoch updates of the stochastic method of
// Section 5.1, Eq. 5, grouped into mini-batches): the template's cells are
// dealt into B batches by a hash of their template position, and each epoch
// takes one batch-restricted step per batch, in batch order.
//
// The batch of cell (a, b) (row a of I, column b of J) is
// splitmix64(seed ^ (a << 32 | b)) mod B, where splitmix64 is the output
// function of Steele, Lea and Flood's SplitMix64 generator (2014): add the
// golden-ratio increment 0x9E3779B97F4A7C15, then xor-shift 30 and multiply
// by 0xBF58476D1CE4E5B9, xor-shift 27 and multiply by 0x94D049BB133111EB,
// xor-shift 31.
//
// Each side's stream gets a batch-major copy: a stable sort on the key
// batch * rows + owner row keeps the cells of one batch bucketed by owner row
// in template order, so batch beta of side s is an ordinary bucketed stream
// with pointers ptr + beta * rows (rows + 1 of them, the last shared with the
// next batch) and the item pass runs on it unchanged.
#include <algorithm>

#include "internal.h"

namespace tsid {

namespace {

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// One wave per owner row; its lanes take the row's cells in strides of 64.
__global__ __launch_bounds__(256) void k_batch_keys(const int2 *stream, const int64_t *ptr, int32_t rows,
                                                    int side, uint64_t seed, uint32_t n_batches,
                                                    uint64_t *keys, uint32_t *vals) {
    const int64_t x = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (x >= rows) return;
    const int lane = threadIdx.x & 63;
    const int64_t b0 = ptr[x], b1 = ptr[x + 1];
    for (int64_t j = b0 + lane; j < b1; j += 64) {
        const uint32_t other = (uint32_t)stream[j].x;
        const uint64_t a = side ? other : (uint64_t)x, b = side ? (uint64_t)x : other;
        const uint64_t beta = splitmix64(seed ^ ((a << 32) | b)) % n_batches;
        keys[j] = beta * (uint64_t)rows + (uint64_t)x;
        vals[j] = (uint32_t)j;
    }
}

__global__ __launch_bounds__(256) void k_gather_stream(const int2 *in, const uint32_t *idx, int64_t n, int2 *out) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += (int64_t)gridDim.x * blockDim.x)
        out[j] = in[idx[j]];
}

}  // namespace

void batch_keys(const int2 *stream, const int64_t *ptr, int32_t rows, int side, uint64_t seed, int32_t n_batches,
                uint64_t *keys, uint32_t *vals, hipStream_t s) {
    if (rows <= 0) return;
    hipLaunchKernelGGL(k_batch_keys, dim3((unsigned)ceil_div(rows, 4)), dim3(256), 0, s, stream, ptr, rows, side,
                       seed, (uint32_t)n_batches, keys, vals);
    TSID_HIP(hipGetLastError());
}

void gather_stream(const int2 *in, const uint32_t *idx, int64_t n, int2 *out, hipStream_t s) {
    if (n <= 0) return;
    const int64_t blocks = std::min<int64_t>((n + 255) / 256, 65536);
    hipLaunchKernelGGL(k_gather_stream, dim3((unsigned)blocks), dim3(256), 0, s, in, idx, n, out);
    TSID_HIP(hipGetLastError());
}

}  // namespace tsid
