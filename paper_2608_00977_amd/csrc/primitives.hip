// Index-building primitives for the resident template (Section 3.2; Section
// 5.1 "Sampling the TSID Template Submatrix"): exclusive scans, a stable LSD
// radix sort for the row and column buckets, the order-preserving filter of
// Omega to Omega*, bucket pointers and the per-bucket work plan.
//
// Everything here is deterministic: counts may use LDS atomics, but every
// output position comes from prefix sums over a fixed element order, so the
// buckets are bit-identical from run to run.
#include "internal.h"

namespace tsid {

namespace {

constexpr int kThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kThreads * kScanItems;  // 2048
constexpr int kSortItems = 16;
constexpr int kSortTile = kThreads * kSortItems;  // 4096
constexpr int kFiltItems = 16;
constexpr int kFiltTile = kThreads * kFiltItems;  // 4096

// Exclusive scan of one value per thread over the 256-thread block; returns
// the exclusive prefix and sets `total`.  Uses `lds` (256 entries).
__device__ uint32_t block_scan_excl(uint32_t v, uint32_t *lds, uint32_t &total) {
    const int t = threadIdx.x;
    lds[t] = v;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        uint32_t add = t >= off ? lds[t - off] : 0u;
        __syncthreads();
        lds[t] += add;
        __syncthreads();
    }
    uint32_t incl = lds[t];
    total = lds[kThreads - 1];
    __syncthreads();
    return incl - v;
}

__global__ __launch_bounds__(kThreads) void k_scan_reduce(const uint32_t *in, int64_t n,
                                                          uint32_t *sums) {
    __shared__ uint32_t lds[kThreads];
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    uint32_t s = 0;
    for (int it = 0; it < kScanItems; ++it) {
        int64_t j = base + (int64_t)it * kThreads + threadIdx.x;
        if (j < n) s += in[j];
    }
    uint32_t total;
    block_scan_excl(s, lds, total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void k_scan_apply(const uint32_t *in, uint32_t *out,
                                                         int64_t n, const uint32_t *block_offs,
                                                         uint32_t *total_out) {
    __shared__ uint32_t tile[kScanTile];
    __shared__ uint32_t lds[kThreads];
    const int64_t base = (int64_t)blockIdx.x * kScanTile;
    for (int it = 0; it < kScanItems; ++it) {
        int64_t j = base + (int64_t)it * kThreads + threadIdx.x;
        tile[it * kThreads + threadIdx.x] = j < n ? in[j] : 0u;
    }
    __syncthreads();
    uint32_t loc[kScanItems];
    uint32_t s = 0;
    for (int it = 0; it < kScanItems; ++it) {
        loc[it] = s;
        s += tile[threadIdx.x * kScanItems + it];
    }
    uint32_t total;
    uint32_t pre = block_scan_excl(s, lds, total);
    uint32_t off = block_offs ? block_offs[blockIdx.x] : 0u;
    for (int it = 0; it < kScanItems; ++it) tile[threadIdx.x * kScanItems + it] = off + pre + loc[it];
    __syncthreads();
    for (int it = 0; it < kScanItems; ++it) {
        int64_t j = base + (int64_t)it * kThreads + threadIdx.x;
        if (j < n) out[j] = tile[it * kThreads + threadIdx.x];
    }
    if (total_out && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *total_out = off + total;
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n;
         j += (int64_t)gridDim.x * blockDim.x)
        p[j] = v;
}

__global__ void k_scatter_map(const int32_t *ids, int32_t count, int32_t *map) {
    int64_t a = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (a < count) map[ids[a]] = (int32_t)a;
}

// ---------------------------------------------------------------- radix sort

// Input already in key order: *unsorted stays 0 and the passes do nothing
// (see radix_sort).
__global__ void k_keys_unsorted(const uint64_t *keys, int64_t n, uint32_t *unsorted) {
    bool bad = false;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x + 1; j < n;
         j += (int64_t)gridDim.x * blockDim.x)
        bad |= keys[j - 1] > keys[j];
    if (bad) *unsorted = 1u;
}

__global__ __launch_bounds__(kThreads) void k_radix_hist(const uint64_t *keys, int64_t n, int shift,
                                                         uint32_t *counts, int nb, const uint32_t *unsorted) {
    if (unsorted && *unsorted == 0u) return;
    __shared__ uint32_t h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int it = 0; it < kSortItems; ++it) {
        int64_t j = base + (int64_t)it * kThreads + threadIdx.x;
        if (j < n) atomicAdd(&h[(uint32_t)(keys[j] >> shift) & 255u], 1u);
    }
    __syncthreads();
    counts[(int64_t)threadIdx.x * nb + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter: elements are ranked in index order (round, wave, lane).
// With unsorted pointing at 0 (input in key order) the pass only copies its
// tile when copy_if_sorted is set (the last of an odd number of passes, whose
// result the caller expects in the other buffer).
__global__ __launch_bounds__(kThreads) void k_radix_scatter(const uint64_t *kin, const uint32_t *vin,
                                                            uint64_t *kout, uint32_t *vout,
                                                            int64_t n, int shift,
                                                            const uint32_t *offs, int nb,
                                                            const uint32_t *unsorted, int copy_if_sorted) {
    __shared__ uint32_t s_base[256];
    __shared__ uint32_t s_cnt[4][256];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    if (unsorted && *unsorted == 0u) {
        if (copy_if_sorted) {
            for (int it = 0; it < kSortItems; ++it) {
                const int64_t j = (int64_t)blockIdx.x * kSortTile + (int64_t)it * kThreads + t;
                if (j < n) {
                    kout[j] = kin[j];
                    vout[j] = vin[j];
                }
            }
        }
        return;
    }
    s_base[t] = offs[(int64_t)t * nb + blockIdx.x];
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t base = (int64_t)blockIdx.x * kSortTile;
    for (int it = 0; it < kSortItems; ++it) {
        s_cnt[0][t] = 0;
        s_cnt[1][t] = 0;
        s_cnt[2][t] = 0;
        s_cnt[3][t] = 0;
        __syncthreads();
        const int64_t j = base + (int64_t)it * kThreads + t;
        const bool valid = j < n;
        const uint64_t key = valid ? kin[j] : 0ull;
        const uint32_t val = valid ? vin[j] : 0u;
        const uint32_t d = (uint32_t)(key >> shift) & 255u;
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bb = __ballot(bit);
            peers &= bit ? bb : ~bb;
        }
        const uint32_t rank = (uint32_t)__popcll(peers & lt);
        if (valid && rank == 0) s_cnt[w][d] = (uint32_t)__popcll(peers);
        __syncthreads();
        if (valid) {
            uint32_t pos = s_base[d] + rank;
            for (int ww = 0; ww < w; ++ww) pos += s_cnt[ww][d];
            kout[pos] = key;
            vout[pos] = val;
        }
        __syncthreads();
        s_base[t] += s_cnt[0][t] + s_cnt[1][t] + s_cnt[2][t] + s_cnt[3][t];
        __syncthreads();
    }
}

// ------------------------------------------------------------------ filter

__global__ __launch_bounds__(kThreads) void k_filter_count(const int32_t *u, const int32_t *i,
                                                           const float *r, int64_t S,
                                                           const int32_t *row_map,
                                                           const int32_t *col_map, int64_t m,
                                                           int64_t n, uint32_t *bcnt, int32_t *err) {
    __shared__ uint32_t lds[kThreads];
    const int64_t base = (int64_t)blockIdx.x * kFiltTile;
    uint32_t c = 0;
    for (int it = 0; it < kFiltItems; ++it) {
        const int64_t j = base + (int64_t)it * kThreads + threadIdx.x;
        if (j >= S) break;
        const int32_t uu = u[j], ii = i[j];
        if (uu < 0 || uu >= m || ii < 0 || ii >= n) {
            err[ERR_RANGE] = 1;
            continue;
        }
        if (row_map[uu] >= 0 && col_map[ii] >= 0) {
            ++c;
            if (!__builtin_isfinite(r[j])) err[ERR_INVAL] = 1;
        }
    }
    uint32_t total;
    block_scan_excl(c, lds, total);
    if (threadIdx.x == 0) bcnt[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void k_filter_write(
    const int32_t *u, const int32_t *i, const float *r, int64_t S, const int32_t *row_map,
    const int32_t *col_map, int64_t m, int64_t n, const uint32_t *boffs, int64_t base_out,
    int bits_b, uint64_t *out_key, uint32_t *out_val) {
    __shared__ uint32_t s_w[4];
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t base = (int64_t)blockIdx.x * kFiltTile;
    int64_t run = base_out + boffs[blockIdx.x];
    for (int it = 0; it < kFiltItems; ++it) {
        const int64_t j = base + (int64_t)it * kThreads + t;
        int32_t a = -1, b = -1;
        if (j < S) {
            const int32_t uu = u[j], ii = i[j];
            if (uu >= 0 && uu < m && ii >= 0 && ii < n) {
                a = row_map[uu];
                b = col_map[ii];
            }
        }
        const bool keep = a >= 0 && b >= 0;
        const uint64_t bal = __ballot(keep);
        if (lane == 0) s_w[w] = (uint32_t)__popcll(bal);
        __syncthreads();
        if (keep) {
            int64_t pos = run + __popcll(bal & lt);
            for (int ww = 0; ww < w; ++ww) pos += s_w[ww];
            out_key[pos] = ((uint64_t)(uint32_t)a << bits_b) | (uint32_t)b;
            out_val[pos] = __float_as_uint(r[j]);
        }
        run += s_w[0] + s_w[1] + s_w[2] + s_w[3];
        __syncthreads();
    }
}

// ------------------------------------------------------------- bucket views

__global__ void k_keys_to_stream(const uint64_t *keys, const uint32_t *vals, int64_t n, int low_bits,
                                 int2 *stream, int32_t *err) {
    const uint64_t mask = (low_bits >= 64) ? ~0ull : ((1ull << low_bits) - 1ull);
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n;
         j += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t k = keys[j];
        stream[j] = make_int2((int)(uint32_t)(k & mask), (int)vals[j]);
        if (j > 0 && keys[j - 1] == k) err[ERR_DUP] = 1;
    }
}

// Global cell keys u * n + i of a piece of Omega, from offset on.
__global__ void k_cell_keys(const int32_t *u, const int32_t *i, int64_t len, int64_t n, uint64_t *keys,
                            uint32_t *vals) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < len;
         j += (int64_t)gridDim.x * blockDim.x) {
        keys[j] = (uint64_t)(uint32_t)u[j] * (uint64_t)n + (uint64_t)(uint32_t)i[j];
        vals[j] = 0u;
    }
}

// Equal neighbours in sorted keys: a repeated cell.
__global__ void k_adjacent_equal(const uint64_t *keys, int64_t n, int32_t *err) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x + 1; j < n;
         j += (int64_t)gridDim.x * blockDim.x)
        if (keys[j - 1] == keys[j]) err[ERR_DUP] = 1;
}

__global__ void k_ptr_from_keys(const uint64_t *keys, int64_t n, int32_t rows, int low_bits,
                                int64_t *ptr) {
    const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (x > rows) return;
    const uint64_t target = (uint64_t)x << low_bits;
    int64_t lo = 0, hi = n;  // first position with key >= target
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if (keys[mid] < target) lo = mid + 1;
        else hi = mid;
    }
    ptr[x] = lo;
}

__global__ void k_swap_key_halves(const uint64_t *keys, int64_t n, int lo_bits, int hi_bits,
                                  uint64_t *out) {
    const uint64_t mask = (1ull << lo_bits) - 1ull;
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n;
         j += (int64_t)gridDim.x * blockDim.x) {
        const uint64_t k = keys[j];
        out[j] = ((k & mask) << hi_bits) | (k >> lo_bits);
    }
}

__global__ void k_chunk_keys(const int32_t *fixed_id, const int32_t *free_id, const float *r,
                             int64_t nnz, int64_t n_fixed, int32_t n_free, int bits_fixed,
                             uint64_t *keys, uint32_t *vals, int32_t *err) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < nnz;
         j += (int64_t)gridDim.x * blockDim.x) {
        int32_t fx = fixed_id[j], fr = free_id[j];
        if (fx < 0 || fx >= n_fixed || fr < 0 || fr >= n_free) {
            err[ERR_RANGE] = 1;
            fx = 0;
            fr = 0;
        }
        keys[j] = ((uint64_t)(uint32_t)fr << bits_fixed) | (uint32_t)fx;
        vals[j] = __float_as_uint(r[j]);
    }
}

__global__ void k_plan_count(const int64_t *ptr, int32_t rows, int32_t E, uint32_t *nparts) {
    const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= rows) return;
    const int64_t deg = ptr[x + 1] - ptr[x];
    nparts[x] = deg <= E ? 1u : (uint32_t)((deg + E - 1) / E);
}

__global__ void k_plan_fill(const uint32_t *item_off, int32_t rows, int32_t *items) {
    const int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (x >= rows) return;
    for (uint32_t it = item_off[x]; it < item_off[x + 1]; ++it) items[it] = (int32_t)x;
}

int grid_for(int64_t n, int threads, int cap = 65536) {
    int64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    return (int)(g > cap ? cap : g);
}

}  // namespace

// --------------------------------------------------------------- host side

size_t scan_scratch_elems(int64_t n) {
    size_t total = 0;
    while (n > kScanTile) {
        const int64_t nb = (n + kScanTile - 1) / kScanTile;
        total += 2 * (size_t)nb;
        n = nb;
    }
    return total + 1;
}

void scan_u32(const uint32_t *in, uint32_t *out, int64_t n, uint32_t *total, uint32_t *scratch,
              hipStream_t s) {
    if (n <= 0) {
        if (total) TSID_HIP(hipMemsetAsync(total, 0, sizeof(uint32_t), s));
        return;
    }
    const int nb = ceil_div(n, kScanTile);
    if (nb == 1) {
        k_scan_apply<<<1, kThreads, 0, s>>>(in, out, n, nullptr, total);
        TSID_HIP(hipGetLastError());
        return;
    }
    uint32_t *sums = scratch, *offs = scratch + nb;
    k_scan_reduce<<<nb, kThreads, 0, s>>>(in, n, sums);
    TSID_HIP(hipGetLastError());
    scan_u32(sums, offs, nb, nullptr, scratch + 2 * (size_t)nb, s);
    k_scan_apply<<<nb, kThreads, 0, s>>>(in, out, n, offs, total);
    TSID_HIP(hipGetLastError());
}

size_t radix_scratch_elems(int64_t n) {
    const int64_t nb = (n + kSortTile - 1) / kSortTile;
    const int64_t counts = 256 * (nb > 0 ? nb : 1);
    return (size_t)counts + scan_scratch_elems(counts);
}

bool radix_sort(uint64_t *keys, uint32_t *vals, uint64_t *keys_alt, uint32_t *vals_alt, int64_t n,
                int nbits, uint32_t *scratch, hipStream_t s, const uint32_t *unsorted) {
    if (n <= 1) return false;
    const int nb = ceil_div(n, kSortTile);
    const int64_t nc = 256 * (int64_t)nb;
    uint32_t *counts = scratch, *scan_tmp = scratch + nc;
    const int passes = (nbits + 7) / 8;
    bool alt = false;
    for (int p = 0; p < passes; ++p) {
        const int shift = 8 * p;
        const uint64_t *kin = alt ? keys_alt : keys;
        const uint32_t *vin = alt ? vals_alt : vals;
        uint64_t *kout = alt ? keys : keys_alt;
        uint32_t *vout = alt ? vals : vals_alt;
        k_radix_hist<<<nb, kThreads, 0, s>>>(kin, n, shift, counts, nb, unsorted);
        TSID_HIP(hipGetLastError());
        scan_u32(counts, counts, nc, nullptr, scan_tmp, s);  // (its values unused when the passes skip)
        const int copy_if_sorted = (p == passes - 1) && (passes & 1);
        k_radix_scatter<<<nb, kThreads, 0, s>>>(kin, vin, kout, vout, n, shift, counts, nb, unsorted,
                                                copy_if_sorted);
        TSID_HIP(hipGetLastError());
        alt = !alt;
    }
    return alt;
}

void keys_unsorted(const uint64_t *keys, int64_t n, uint32_t *unsorted, hipStream_t s) {
    fill_u32(unsorted, 1, 0u, s);
    if (n <= 1) return;
    k_keys_unsorted<<<grid_for(n, 256), 256, 0, s>>>(keys, n, unsorted);
    TSID_HIP(hipGetLastError());
}

void fill_i32(int32_t *p, int64_t n, int32_t v, hipStream_t s) {
    if (n <= 0) return;
    k_fill_i32<<<grid_for(n, 256), 256, 0, s>>>(p, n, v);
    TSID_HIP(hipGetLastError());
}

void fill_u32(uint32_t *p, int64_t n, uint32_t v, hipStream_t s) {
    fill_i32(reinterpret_cast<int32_t *>(p), n, (int32_t)v, s);
}

void fill_f32(float *p, int64_t n, float v, hipStream_t s) {
    fill_i32(reinterpret_cast<int32_t *>(p), n, (int32_t)__builtin_bit_cast(uint32_t, v), s);
}

void scatter_map(const int32_t *ids, int32_t count, int32_t *map, hipStream_t s) {
    if (count <= 0) return;
    k_scatter_map<<<ceil_div(count, 256), 256, 0, s>>>(ids, count, map);
    TSID_HIP(hipGetLastError());
}

int filter_blocks(int64_t S) { return ceil_div(S > 0 ? S : 1, kFiltTile); }

void filter_count(const int32_t *u, const int32_t *i, const float *r, int64_t S,
                  const int32_t *row_map, const int32_t *col_map, int64_t m, int64_t n,
                  uint32_t *bcnt, int32_t *err, hipStream_t s) {
    if (S <= 0) return;
    k_filter_count<<<filter_blocks(S), kThreads, 0, s>>>(u, i, r, S, row_map, col_map, m, n, bcnt,
                                                         err);
    TSID_HIP(hipGetLastError());
}

void filter_write(const int32_t *u, const int32_t *i, const float *r, int64_t S,
                  const int32_t *row_map, const int32_t *col_map, int64_t m, int64_t n,
                  const uint32_t *boffs, int64_t base, int bits_b, uint64_t *out_key,
                  uint32_t *out_val, hipStream_t s) {
    if (S <= 0) return;
    k_filter_write<<<filter_blocks(S), kThreads, 0, s>>>(u, i, r, S, row_map, col_map, m, n, boffs,
                                                         base, bits_b, out_key, out_val);
    TSID_HIP(hipGetLastError());
}

void keys_to_stream(const uint64_t *keys, const uint32_t *vals, int64_t n, int low_bits,
                    int2 *stream, int32_t *err, hipStream_t s) {
    if (n <= 0) return;
    k_keys_to_stream<<<grid_for(n, 256), 256, 0, s>>>(keys, vals, n, low_bits, stream, err);
    TSID_HIP(hipGetLastError());
}

void cell_keys(const int32_t *u, const int32_t *i, int64_t len, int64_t n, uint64_t *keys, uint32_t *vals,
               hipStream_t s) {
    if (len <= 0) return;
    k_cell_keys<<<grid_for(len, 256), 256, 0, s>>>(u, i, len, n, keys, vals);
    TSID_HIP(hipGetLastError());
}

void adjacent_equal(const uint64_t *keys, int64_t n, int32_t *err, hipStream_t s) {
    if (n <= 1) return;
    k_adjacent_equal<<<grid_for(n, 256), 256, 0, s>>>(keys, n, err);
    TSID_HIP(hipGetLastError());
}

void ptr_from_keys(const uint64_t *keys, int64_t n, int32_t rows, int low_bits, int64_t *ptr,
                   hipStream_t s) {
    k_ptr_from_keys<<<ceil_div((int64_t)rows + 1, 256), 256, 0, s>>>(keys, n, rows, low_bits, ptr);
    TSID_HIP(hipGetLastError());
}

void swap_key_halves(const uint64_t *keys, int64_t n, int lo_bits, int hi_bits, uint64_t *out,
                     hipStream_t s) {
    if (n <= 0) return;
    k_swap_key_halves<<<grid_for(n, 256), 256, 0, s>>>(keys, n, lo_bits, hi_bits, out);
    TSID_HIP(hipGetLastError());
}

void chunk_keys(const int32_t *fixed_id, const int32_t *free_id, const float *r, int64_t nnz,
                int64_t n_fixed, int32_t n_free, int bits_fixed, uint64_t *keys, uint32_t *vals,
                int32_t *err, hipStream_t s) {
    if (nnz <= 0) return;
    k_chunk_keys<<<grid_for(nnz, 256), 256, 0, s>>>(fixed_id, free_id, r, nnz, n_fixed, n_free,
                                                    bits_fixed, keys, vals, err);
    TSID_HIP(hipGetLastError());
}

void plan_items(const int64_t *ptr, int32_t rows, int32_t E, uint32_t *item_off, int32_t *items,
                uint32_t *nparts_scratch, uint32_t *scan_scratch, hipStream_t s) {
    if (rows <= 0) {
        TSID_HIP(hipMemsetAsync(item_off, 0, sizeof(uint32_t), s));
        return;
    }
    k_plan_count<<<ceil_div(rows, 256), 256, 0, s>>>(ptr, rows, E, nparts_scratch);
    TSID_HIP(hipGetLastError());
    scan_u32(nparts_scratch, item_off, rows, item_off + rows, scan_scratch, s);
    k_plan_fill<<<ceil_div(rows, 256), 256, 0, s>>>(item_off, rows, items);
    TSID_HIP(hipGetLastError());
}

}  // namespace tsid
