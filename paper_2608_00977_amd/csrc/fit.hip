// Template-fit kernels (Stage I, Section 5.1): per observed cell the residual
// e = r - p_a . q_b, the per-cell gradients of Eqs. 3-4 aggregated into the
// owning factor row, and the row update of Eq. 5 with the asymmetric clip of
// Section 5.3.  The same kernels run the one-sided extension steps of Section
// 5.2 (owner = free rows, gathered side = fixed factors).
//
// Layout and mapping (gfx950, wave64):
//  * A bucketed stream holds one 8-byte {other id, value} record per cell,
//    grouped by the owning row (CSR for the P pass, CSC for the Q pass) and
//    read once per pass with non-temporal loads.
//  * A bucket is cut into work items of at most E cells.  Each item belongs
//    to a group of G = K / V lanes; lane g of the group holds V coordinates of
//    the owner row in registers: [g*V, g*V + V) when V coordinates fill one
//    16-byte chunk of the gathered table, else chunks g, g + G, g + 2G, ...
//    (so that each gather instruction reads consecutive bytes; see Lanes).
//  * Per cell the group gathers the other factor row (16 bytes per lane and
//    chunk), forms the dot product with a DPP butterfly inside the group (all
//    lanes end with the same bits), and accumulates e * q into its registers.
//  * The aggregated gradient goes straight to the owner row when the bucket is
//    one item; split buckets leave one partial sum per item and a fixup kernel
//    adds the parts in item order.  No atomics touch factor or gradient memory,
//    so results are bitwise reproducible.
//  * bf16 mode: the gathered side is a bf16 copy (2 bytes per coordinate, dots
//    by v_dot2_f32_bf16 with fp32 accumulation); the owner row's fp32 master
//    takes the update and a round-to-nearest-even bf16 copy is written beside it.
#include <hip/hip_ext.h>

#include "internal.h"

namespace tsid {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, true));
}

// Sum over an aligned group of G lanes (G <= 16: the group lies inside one DPP
// row).  Butterfly pairs: quad_perm [1,0,3,2], quad_perm [2,3,0,1],
// row_half_mirror, row_mirror.  IEEE addition commutes, so every lane of the
// group ends with the same bits.
template <int G>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (G >= 2) x += dpp<0xB1>(x);
    if constexpr (G >= 4) x += dpp<0x4E>(x);
    if constexpr (G >= 8) x += dpp<0x141>(x);
    if constexpr (G >= 16) x += dpp<0x140>(x);
    return x;
}

// Value of lane `t` of this lane's aligned group of G lanes, for every lane
// of the group: ds_swizzle in bit mode, new lane = (lane & ~(G-1)) | t within
// each 32-lane half (and_mask in bits 0-4, or_mask in bits 5-9).
template <int CTRL>
__device__ __forceinline__ int dpp_i(int x) {
    return __builtin_amdgcn_update_dpp(0, x, CTRL, 0xF, 0xF, true);
}

template <int G>
__device__ __forceinline__ int group_bcast(int v, int t) {
    if constexpr (G == 1) {
        return v;
    } else if constexpr (G == 2) {
        // DPP quad_perm [t, t, 2+t, 2+t]: a VALU move, no LDS traffic
        return t == 0 ? dpp_i<0xA0>(v) : dpp_i<0xF5>(v);
    } else if constexpr (G == 4) {
        // DPP quad_perm [t, t, t, t]
        switch (t) {
            case 0: return dpp_i<0x00>(v);
            case 1: return dpp_i<0x55>(v);
            case 2: return dpp_i<0xAA>(v);
            default: return dpp_i<0xFF>(v);
        }
    } else {
        static_assert(G <= 32, "groups live inside one 32-lane half");
        int out = v;
        // t is a compile-time constant after unrolling; the switch keeps the
        // swizzle pattern an immediate.
        switch (t) {
#define TSID_BCAST_CASE(T_) \
    case T_: out = __builtin_amdgcn_ds_swizzle(v, (0x1F & ~(G - 1)) | ((T_) << 5)); break;
            TSID_BCAST_CASE(0) TSID_BCAST_CASE(1) TSID_BCAST_CASE(2) TSID_BCAST_CASE(3)
            TSID_BCAST_CASE(4) TSID_BCAST_CASE(5) TSID_BCAST_CASE(6) TSID_BCAST_CASE(7)
            TSID_BCAST_CASE(8) TSID_BCAST_CASE(9) TSID_BCAST_CASE(10) TSID_BCAST_CASE(11)
            TSID_BCAST_CASE(12) TSID_BCAST_CASE(13) TSID_BCAST_CASE(14) TSID_BCAST_CASE(15)
#undef TSID_BCAST_CASE
            default: break;
        }
        return out;
    }
}

// IEEE round-to-nearest-even of fp32 to bf16 (NaN stays NaN).
__device__ __forceinline__ uint32_t bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

template <int V>
__device__ __forceinline__ void load_f32(const float *p, float (&x)[V]) {
    const float4 *q = reinterpret_cast<const float4 *>(p);
#pragma unroll
    for (int c = 0; c < V / 4; ++c) {
        const float4 t = q[c];
        x[4 * c + 0] = t.x;
        x[4 * c + 1] = t.y;
        x[4 * c + 2] = t.z;
        x[4 * c + 3] = t.w;
    }
}

template <int V>
__device__ __forceinline__ void store_f32(float *p, const float (&x)[V]) {
    float4 *q = reinterpret_cast<float4 *>(p);
#pragma unroll
    for (int c = 0; c < V / 4; ++c) q[c] = make_float4(x[4 * c], x[4 * c + 1], x[4 * c + 2], x[4 * c + 3]);
}

// The coordinates a lane holds.  A row of the gathered table is read in
// 16-byte chunks (Q coordinates: 8 in bf16, 4 in fp32); lane lg of a group of
// G lanes holds V / Q of them, its n-th being chunk n G + lg of the row, so
// that one gather instruction of a group reads G * 16 consecutive bytes
// (whole 128-byte lines at G = 8) instead of a strided part of every line of
// the row.  Element n Q + j of a lane's arrays is coordinate coord(lg, n) + j;
// with one chunk per lane this is the plain split lg V .. lg V + V - 1.
template <int G, int V, bool BF16>
struct Lanes {
    static constexpr int Q = BF16 ? 8 : 4;
    static constexpr int N = V / Q;
    static_assert(V % Q == 0, "a lane holds whole 16-byte chunks");
    static __device__ __forceinline__ int coord(int lg, int n) { return (n * G + lg) * Q; }
};

// This lane's coordinates of an fp32 row (row points at coordinate 0).
template <int G, int V, bool BF16>
__device__ __forceinline__ void load_coords(const float *row, int lg, float (&x)[V]) {
    using L = Lanes<G, V, BF16>;
#pragma unroll
    for (int n = 0; n < L::N; ++n) {
#pragma unroll
        for (int w = 0; w < L::Q / 4; ++w) {
            const float4 t = *reinterpret_cast<const float4 *>(row + L::coord(lg, n) + 4 * w);
            x[n * L::Q + 4 * w + 0] = t.x;
            x[n * L::Q + 4 * w + 1] = t.y;
            x[n * L::Q + 4 * w + 2] = t.z;
            x[n * L::Q + 4 * w + 3] = t.w;
        }
    }
}

template <int G, int V, bool BF16>
__device__ __forceinline__ void store_coords(float *row, int lg, const float (&x)[V]) {
    using L = Lanes<G, V, BF16>;
#pragma unroll
    for (int n = 0; n < L::N; ++n) {
#pragma unroll
        for (int w = 0; w < L::Q / 4; ++w) {
            const int e = n * L::Q + 4 * w;
            *reinterpret_cast<float4 *>(row + L::coord(lg, n) + 4 * w) = make_float4(x[e], x[e + 1], x[e + 2], x[e + 3]);
        }
    }
}

// Cells a lane group takes per chunk (rounded to a multiple of the group).
#ifndef TSID_CELLS_PER_GROUP
#define TSID_CELLS_PER_GROUP 8
#endif
// 1: stream loads carry the non-temporal hint.
#ifndef TSID_STREAM_NT
#define TSID_STREAM_NT 0
#endif

__device__ __forceinline__ int2 load_cell(const int2 *p) {
#if TSID_STREAM_NT
    const long long v = __builtin_nontemporal_load(reinterpret_cast<const long long *>(p));
#else
    const long long v = *reinterpret_cast<const long long *>(p);
#endif
    return make_int2((int)(uint32_t)(unsigned long long)v, (int)(uint32_t)((unsigned long long)v >> 32));
}

__device__ __forceinline__ bool skip_epoch(const PassArgs &A) {
    if (!A.skip_after_nonfinite) return false;
    const int32_t f = A.err[ERR_NONFINITE];
    return f != 0 && f - 1 < A.epoch;
}

// Row update of Eq. 5 (descent on Eqs. 3-4 summed), optional 1/max(1, deg)
// normalisation and the Section 5.3 clip, for this lane's V coordinates.
template <int G, int V, bool BF16>
__device__ __forceinline__ void finalize_row(const PassArgs &A, int row, int lg, const float (&x)[V],
                                             const float (&acc_in)[V], int64_t deg) {
    if (A.partial_out) {  // a row block's pass: the sum only, the update comes later
        store_coords<G, V, BF16>(A.partial_out + (int64_t)row * (G * V), lg, acc_in);
        return;
    }
    float acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = acc_in[v];
    if (A.dptr) {
        // dense head tiles: the stream holds the other cells only; the degree
        // counts every cell and the tiles' gradient sums are added here
        deg = A.dptr[row + 1] - A.dptr[row];
        if (A.gd_tile_ptr[(row >> 4) + 1] > A.gd_tile_ptr[row >> 4]) {
            float g[V];
            load_coords<G, V, BF16>(A.gd + (int64_t)row * (G * V), lg, g);
#pragma unroll
            for (int v = 0; v < V; ++v) acc[v] += g[v];
        }
    }
    const float s = A.degree ? 1.0f / (float)(deg > 1 ? deg : 1) : 1.0f;
    const bool keep = A.keep_empty && deg == 0;
    float gxv[V];
#pragma unroll
    for (int v = 0; v < V; ++v) gxv[v] = 0.f;
    if (A.gx) load_coords<G, V, BF16>(A.gx + (int64_t)row * (G * V), lg, gxv);
    float xn[V];
    bool bad = false;
    float nrm = 0.f;
#pragma unroll
    for (int v = 0; v < V; ++v) {
        float d;
        if (A.clip == 2) {
            d = s * acc[v];  // the cells' clipped directions (per-entry order)
        } else {
            float g = 2.0f * A.lam * x[v] - 2.0f * acc[v];
            if (A.gx) g += A.gx_scale * gxv[v];
            d = clipped_step(g, s, A.clip, A.xi);
        }
        xn[v] = keep ? x[v] : x[v] + A.lr * d;
        bad |= !__builtin_isfinite(xn[v]);
        nrm += x[v] * x[v];
    }
    const int64_t off = (int64_t)row * (G * V);
    store_coords<G, V, BF16>(A.Xn + off, lg, xn);
    if constexpr (BF16) {
        static_assert(V % 8 == 0, "bf16 rows hold a multiple of 8 coordinates per lane");
        if (A.Xn_b) {
#pragma unroll
            for (int c = 0; c < V / 8; ++c) {
                uint32_t w[4];
#pragma unroll
                for (int p = 0; p < 4; ++p)
                    w[p] = bf16_bits(xn[8 * c + 2 * p]) | (bf16_bits(xn[8 * c + 2 * p + 1]) << 16);
                *reinterpret_cast<uint4 *>(A.Xn_b + off + Lanes<G, V, true>::coord(lg, c)) =
                    make_uint4(w[0], w[1], w[2], w[3]);
            }
        }
    }
    nrm = group_sum<G>(nrm);
    if (lg == 0 && A.norm) A.norm[row] = nrm;
    if (bad) A.err[ERR_NONFINITE] = A.epoch + 1;
}

// Gathers of the other factor.  Within the template (tables below 4 GiB) they
// are raw buffer loads: one 32-bit offset register per gather instead of a
// 64-bit address, and the hardware clamps any offset past the table to zero.
// The extension's fixed table may exceed 4 GiB and uses 64-bit global loads.
struct YTable {
    __amdgpu_buffer_rsrc_t rsrc;
    const char *base;
};

template <bool BUF>
__device__ __forceinline__ YTable make_ytable(const PassArgs &A, int row_bytes) {
    YTable t;
    t.base = static_cast<const char *>(A.Y);
    if constexpr (BUF) {
        // raw buffer, 32-bit data format (descriptor word 3 of the gfx9 family)
        t.rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(A.Y), (short)0,
                                                   (int)(A.y_rows * row_bytes), 0x00020000);
    }
    return t;
}

// 16 bytes of row b of the table at byte offset `col_byte` within the row.
template <bool BUF>
__device__ __forceinline__ uint4 ygather16(const YTable &t, int b, int row_bytes, int col_byte) {
    if constexpr (BUF) {
        return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                             t.rsrc, (unsigned)(b * row_bytes + col_byte), 0, 0));
    } else {
        return *reinterpret_cast<const uint4 *>(t.base + (int64_t)b * row_bytes + col_byte);
    }
}

// Stream layout of a group's walk over its item: cells arrive in blocks of
// SB = G * SPL cells (SPL per lane: lane s holds cells s + c*G, c < SPL),
// and are consumed in chunks of CH cells, CH gathers in flight per lane.
#ifndef TSID_PINGPONG
#define TSID_PINGPONG 0
#endif
#ifndef TSID_CHUNK_BARRIER
#define TSID_CHUNK_BARRIER 0
#endif
#ifndef TSID_STREAM_SPL
#define TSID_STREAM_SPL 16
#endif
template <int G>
constexpr int chunk_cells() {
    return TSID_CELLS_PER_GROUP < G ? G : TSID_CELLS_PER_GROUP;
}
template <int G>
constexpr int block_spl() {  // stream cells per lane per block
    return (G * TSID_STREAM_SPL) < chunk_cells<G>() ? (chunk_cells<G>() / G) : TSID_STREAM_SPL;
}

// One stream block of a work item (SB = G * SPL cells starting at j0).  Per
// chunk of CH cells the group broadcasts each cell's column id and issues
// all CH gathers, then does the arithmetic.  After the gathers of the last
// chunk -- and before its arithmetic -- the group issues the loads of the
// next block's cells into `nxt`: loads retire in issue order, so the slow
// stream loads must come after every gather the arithmetic waits for, and
// issuing them once per block exposes their latency once per SB cells.
// NEXT = false skips those loads (the caller's cells all fit one block).
// PE: the per-entry order of the clipped update -- each cell adds its own
// descent direction 2 e y - 2 lambda x, clipped at xi, instead of e y.
template <int K, int V, bool BF16, bool LOSS_ONLY, bool BUF, bool NEXT = true, int SPL = block_spl<K / V>(),
          bool PE = false>
__device__ __forceinline__ void process_block(const PassArgs &A, const YTable &Yt, int64_t j0,
                                              int64_t end, int64_t last, int lg, const int2 (&cur)[SPL],
                                              int2 (&nxt)[SPL], const float (&x)[V],
                                              const uint32_t (&xp)[V / 2], float (&acc)[V], float &e2) {
    constexpr int G = K / V;
    constexpr int SB = G * SPL;
    constexpr int CH = chunk_cells<G>();
    static_assert(SB % CH == 0, "a stream block holds whole chunks");
    const int64_t left = end - j0;
#pragma unroll
    for (int c0 = 0; c0 < SB; c0 += CH) {
        const bool last_chunk = (c0 + CH == SB);
        if (c0 > 0 && c0 >= left) break;  // the item ends inside this block
#if TSID_CHUNK_BARRIER
        __builtin_amdgcn_sched_barrier(0);  // no hoisting across chunks: fewer live registers
#endif
        if constexpr (BF16) {
            uint32_t yw[CH][V / 2];
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const int b = group_bcast<G>(cur[(c0 + t) / G].x, (c0 + t) % G);
#pragma unroll
                for (int c = 0; c < V / 8; ++c) {
                    const uint4 q = ygather16<BUF>(Yt, b, K * 2, Lanes<G, V, true>::coord(lg, c) * 2);
                    yw[t][4 * c + 0] = q.x;
                    yw[t][4 * c + 1] = q.y;
                    yw[t][4 * c + 2] = q.z;
                    yw[t][4 * c + 3] = q.w;
                }
            }
            if (NEXT && last_chunk) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int c = 0; c < SPL; ++c) {
                    const int64_t jn = j0 + SB + c * G + lg;
                    nxt[c] = load_cell(A.stream + (jn < last ? jn : last));
                }
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const float r = __int_as_float(group_bcast<G>(cur[(c0 + t) / G].y, (c0 + t) % G));
                float d = 0.f;
#pragma unroll
                for (int p = 0; p < V / 2; ++p)
                    d = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, xp[p]),
                                                         __builtin_bit_cast(bf16x2, yw[t][p]), d, false);
                d = group_sum<G>(d);
                const bool in = c0 + t < left;
                const float e = in ? r - d : 0.f;
                if constexpr (!LOSS_ONLY && PE) {
#pragma unroll
                    for (int p = 0; p < V / 2; ++p) {
                        float d0 = 2.0f * e * __uint_as_float(yw[t][p] << 16) - 2.0f * A.lam * x[2 * p];
                        float d1 = 2.0f * e * __uint_as_float(yw[t][p] & 0xffff0000u) - 2.0f * A.lam * x[2 * p + 1];
                        if (d0 > A.xi) d0 = A.xi;
                        if (d1 > A.xi) d1 = A.xi;
                        acc[2 * p] += in ? d0 : 0.f;
                        acc[2 * p + 1] += in ? d1 : 0.f;
                    }
                } else if constexpr (!LOSS_ONLY) {
#pragma unroll
                    for (int p = 0; p < V / 2; ++p) {
                        acc[2 * p] += e * __uint_as_float(yw[t][p] << 16);
                        acc[2 * p + 1] += e * __uint_as_float(yw[t][p] & 0xffff0000u);
                    }
                }
                e2 += e * e;
            }
        } else {
            float y[CH][V];
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const int b = group_bcast<G>(cur[(c0 + t) / G].x, (c0 + t) % G);
#pragma unroll
                for (int c = 0; c < V / 4; ++c) {
                    const uint4 q = ygather16<BUF>(Yt, b, K * 4, Lanes<G, V, false>::coord(lg, c) * 4);
                    y[t][4 * c + 0] = __uint_as_float(q.x);
                    y[t][4 * c + 1] = __uint_as_float(q.y);
                    y[t][4 * c + 2] = __uint_as_float(q.z);
                    y[t][4 * c + 3] = __uint_as_float(q.w);
                }
            }
            if (NEXT && last_chunk) {
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int c = 0; c < SPL; ++c) {
                    const int64_t jn = j0 + SB + c * G + lg;
                    nxt[c] = load_cell(A.stream + (jn < last ? jn : last));
                }
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const float r = __int_as_float(group_bcast<G>(cur[(c0 + t) / G].y, (c0 + t) % G));
                float d = 0.f;
#pragma unroll
                for (int v = 0; v < V; ++v) d += x[v] * y[t][v];
                d = group_sum<G>(d);
                const bool in = c0 + t < left;
                const float e = in ? r - d : 0.f;
                if constexpr (!LOSS_ONLY && PE) {
#pragma unroll
                    for (int v = 0; v < V; ++v) {
                        float dv = 2.0f * e * y[t][v] - 2.0f * A.lam * x[v];
                        if (dv > A.xi) dv = A.xi;
                        acc[v] += in ? dv : 0.f;
                    }
                } else if constexpr (!LOSS_ONLY) {
#pragma unroll
                    for (int v = 0; v < V; ++v) acc[v] += e * y[t][v];
                }
                e2 += e * e;
            }
        }
    }
}

// Waves per SIMD the register allocation must allow (0: compiler's choice).
#ifndef TSID_WAVES_PER_EU
#define TSID_WAVES_PER_EU 0
#endif
#if TSID_WAVES_PER_EU > 0
#define TSID_OCCUPANCY __attribute__((amdgpu_waves_per_eu(TSID_WAVES_PER_EU, TSID_WAVES_PER_EU)))
#else
#define TSID_OCCUPANCY
#endif

// Workgroup `bid` of one side's item pass.
template <int K, int V, bool BF16, bool LOSS_ONLY, bool BUF, bool PE>
__device__ __forceinline__ void item_pass_group(const PassArgs &A, const int64_t bid) {
    constexpr int G = K / V;
    constexpr int NG = 64 / G;
    static_assert(G >= 1 && G <= 16 && (G & (G - 1)) == 0, "group must fit a DPP row");
    if (skip_epoch(A)) return;
    const int lane = threadIdx.x & 63;
    const int grp = lane / G, lg = lane % G;
    const int64_t item = (bid * kWaves + (threadIdx.x >> 6)) * NG + grp;
    const int64_t n_items = A.n_items_dev ? (int64_t)*A.n_items_dev : (int64_t)A.n_items;
    if (item >= n_items) return;  // whole groups leave together
    const int row = A.items[item];  // -1: a pad item that keeps buckets wave-aligned
    uint32_t i0 = 0, i1 = 0;
    int64_t re = 0, beg = 0, end = 0;
    float x[V];
    if (row >= 0) {
        // the bucket's cells split evenly over its items (at most E each)
        i0 = A.item_off[row];
        i1 = A.item_end[row];
        const int64_t rb = A.ptr[row];
        re = A.ptr_end ? A.ptr_end[row] : A.ptr[row + 1];
        const int64_t deg = re - rb, parts = (int64_t)(i1 - i0), q = item - (int64_t)i0;
        beg = rb + q * deg / parts;
        end = rb + (q + 1) * deg / parts;
        const int64_t orow = A.owner_mod ? row % A.owner_mod : row;
        load_coords<G, V, BF16>(A.X + orow * K, lg, x);
    } else {
#pragma unroll
        for (int v = 0; v < V; ++v) x[v] = 0.f;
    }
    uint32_t xp[V / 2] = {};  // bf16 pairs of the owner row (bf16 mode)
    if constexpr (BF16) {
#pragma unroll
        for (int p = 0; p < V / 2; ++p) xp[p] = bf16_bits(x[2 * p]) | (bf16_bits(x[2 * p + 1]) << 16);
    }
    float acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = 0.f;
    float e2 = 0.f;

    // The group walks its cells one stream block at a time (see
    // process_block); two cell buffers alternate so the next block's cells
    // load into the buffer not in use.  Loads past the item's end re-read its
    // last cell (always in bounds and unconditional, so outstanding loads are
    // counted exactly); the slots they fill are masked inside process_block.
    constexpr int SPL = block_spl<G>();
    constexpr int SB = G * SPL;
    const int64_t last = end - 1;
    int2 bufA[SPL], bufB[SPL];
    if (end > beg) {
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int64_t jj = beg + c * G + lg;
            bufA[c] = load_cell(A.stream + (jj < last ? jj : last));
        }
    }
    const YTable Yt = make_ytable<BUF>(A, K * (BF16 ? 2 : 4));
#if TSID_PINGPONG
    for (int64_t j0 = beg; j0 < end; j0 += 2 * SB) {
        process_block<K, V, BF16, LOSS_ONLY, BUF, true, block_spl<K / V>(), PE>(A, Yt, j0, end, last, lg, bufA, bufB, x, xp, acc, e2);
        if (j0 + SB >= end) break;
        process_block<K, V, BF16, LOSS_ONLY, BUF, true, block_spl<K / V>(), PE>(A, Yt, j0 + SB, end, last, lg, bufB, bufA, x, xp, acc,
                                                  e2);
    }
#else
    // One block body per iteration; the block's last stream loads land in
    // bufB and are copied over only after the block's arithmetic, where the
    // next block needs them anyway.
    for (int64_t j0 = beg; j0 < end; j0 += SB) {
        process_block<K, V, BF16, LOSS_ONLY, BUF, true, block_spl<K / V>(), PE>(A, Yt, j0, end, last, lg, bufA, bufB, x, xp, acc, e2);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int c = 0; c < SPL; ++c) bufA[c] = bufB[c];
    }
#endif

    if (A.e2 && lg == 0) A.e2[item] = e2;
    if constexpr (LOSS_ONLY) {
        if (A.norm && row >= 0 && item == (int64_t)i0) {
            float nrm = 0.f;
#pragma unroll
            for (int v = 0; v < V; ++v) nrm += x[v] * x[v];
            nrm = group_sum<G>(nrm);
            if (lg == 0) A.norm[row] = nrm;
        }
    } else {
        // Groups of this wave that hold consecutive items of the same bucket add
        // their partial sums through LDS, in group order, into the segment's
        // first group.  A bucket whose items all sit in this wave is updated
        // here; otherwise the segment leaves one partial sum, at the index of its
        // first item, for the fixup kernel.
        __shared__ float red[kWaves][NG][K];
        __shared__ int seg_row[kWaves][NG];
        const int wv = threadIdx.x >> 6;
        store_f32<V>(&red[wv][grp][lg * V], acc);
        if (lg == 0) seg_row[wv][grp] = row;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // items are in bucket order (pads hold -1), so the group before this one
        // has published its bucket
        const bool head = row >= 0 && ((grp == 0) || (seg_row[wv][grp - 1] != row));
        if (head) {
            int g_end = grp + 1;
            while (g_end < NG && item + (g_end - grp) < n_items && seg_row[wv][g_end] == row) ++g_end;
            for (int g = grp + 1; g < g_end; ++g) {
                float part[V];
                load_f32<V>(&red[wv][g][lg * V], part);
#pragma unroll
                for (int v = 0; v < V; ++v) acc[v] += part[v];
            }
            const int64_t seg_last = item + (g_end - grp) - 1;
            if (item == (int64_t)i0 && seg_last == (int64_t)i1 - 1) {
                finalize_row<G, V, BF16>(A, row, lg, x, acc, re - A.ptr[row]);
            } else {
                store_f32<V>(A.carry + (A.carry_per_wave ? item / NG : item) * K + lg * V, acc);
            }
        }
    }
}

template <int K, int V, bool BF16, bool LOSS_ONLY, bool BUF, bool PE = false>
__global__ __launch_bounds__(kThreads) TSID_OCCUPANCY void k_item_pass(const PassArgs A) {
    item_pass_group<K, V, BF16, LOSS_ONLY, BUF, PE>(A, blockIdx.x);
}

// Both passes of a simultaneous step in one launch: the Q pass reads only the
// old factors, so the b0 workgroups of the P pass (A0) and then those of the
// Q pass (A1) share one grid, and the Q pass's workgroups start as the P
// pass's leave the compute units.
template <int K, int V, bool BF16, bool BUF, bool PE>
__global__ __launch_bounds__(kThreads) TSID_OCCUPANCY void k_item_pass_pair(const PassArgs A0, const PassArgs A1,
                                                                           const int32_t b0) {
    const int b = blockIdx.x;
    if (b < b0)
        item_pass_group<K, V, BF16, false, BUF, PE>(A0, b);
    else
        item_pass_group<K, V, BF16, false, BUF, PE>(A1, b - b0);
}

// The item pass over a plan laid out in workgroup-sized chunks, in the order
// the host chose (sched[w]: the chunk of workgroup w, < 0 for none).  The
// row-blocked Q pass uses it to give each XCD its own block of the gathered
// table: the dispatcher hands workgroups to the XCDs in turn, so workgroup w
// runs on XCD w % 8.
template <int K, int V, bool BF16, bool BUF, bool PE>
__global__ __launch_bounds__(kThreads) TSID_OCCUPANCY void k_item_pass_sched(const PassArgs A, const int32_t *sched) {
    const int32_t chunk = sched[blockIdx.x];
    if (chunk < 0) return;
    item_pass_group<K, V, BF16, false, BUF, PE>(A, chunk);
}

// Split buckets: add the item partial sums in item order, then update the row.
template <int K, int V, bool BF16>
__global__ __launch_bounds__(kThreads) void k_fixup(const PassArgs A) {
    constexpr int G = K / V;
    constexpr int NG = 64 / G;
    if (skip_epoch(A)) return;
    const int lane = threadIdx.x & 63;
    const int grp = lane / G, lg = lane % G;
    const int64_t row = ((int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6)) * NG + grp;
    if (row >= A.rows) return;
    const uint32_t i0 = A.item_off[row], i1 = A.item_end[row];
    // the pass already updated buckets whose items all sat in one wave
    if (i1 - i0 <= 1 || i0 / NG == (i1 - 1) / NG) return;
    float acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = 0.f;
    // one partial sum per wave segment, stored at the segment's first item:
    // the bucket's first item and every later item that starts a wave
    for (uint32_t it = i0; it < i1; it = (it / NG + 1) * NG) {
        float part[V];
        load_f32<V>(A.carry + (int64_t)(A.carry_per_wave ? it / NG : it) * K + lg * V, part);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += part[v];
    }
    float x[V];
    load_coords<G, V, BF16>(A.X + (A.owner_mod ? row % A.owner_mod : row) * K, lg, x);
    finalize_row<G, V, BF16>(A, (int)row, lg, x, acc, A.ptr[row + 1] - A.ptr[row]);
}

// Row-blocked passes.  Bounds of every bucket's runs of other indices per
// block (binary search inside the bucket; one thread per bucket and block).
__global__ void k_block_bounds(const int2 *stream, const int64_t *ptr, int32_t rows, int32_t n_blocks,
                               const int64_t *row_bounds, int64_t *bounds) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)(n_blocks + 1) * rows) return;
    const int64_t j = t / rows, x = t % rows;
    const int64_t target = row_bounds[j];
    int64_t lo = ptr[x], hi = ptr[x + 1];  // first position whose other index >= target
    while (lo < hi) {
        const int64_t mid = lo + ((hi - lo) >> 1);
        if ((int64_t)stream[mid].x < target) lo = mid + 1;
        else hi = mid;
    }
    bounds[t] = lo;
}

// The blocks' partial sums of a row added in block order, then its update
// (one lane group per row, as in k_fixup).
template <int K, int V, bool BF16>
__global__ __launch_bounds__(kThreads) void k_block_combine(const PassArgs A, const float *part, int32_t n_blocks) {
    constexpr int G = K / V;
    constexpr int NG = 64 / G;
    if (skip_epoch(A)) return;
    const int lane = threadIdx.x & 63;
    const int grp = lane / G, lg = lane % G;
    const int64_t row = ((int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6)) * NG + grp;
    if (row >= A.rows) return;
    float acc[V];
    load_coords<G, V, BF16>(part + row * K, lg, acc);
    for (int32_t j = 1; j < n_blocks; ++j) {
        float p[V];
        load_coords<G, V, BF16>(part + ((int64_t)j * A.rows + row) * K, lg, p);
#pragma unroll
        for (int v = 0; v < V; ++v) acc[v] += p[v];
    }
    float x[V];
    load_coords<G, V, BF16>(A.X + row * K, lg, x);
    finalize_row<G, V, BF16>(A, (int)row, lg, x, acc, A.ptr[row + 1] - A.ptr[row]);
}

// One-sided extension steps (Section 5.2, Eq. 6 in factored form), all T of
// them in one launch.  A free row's steps need nothing from other rows, so a
// wave owns one free row (bucket) for the whole run: its NG lane groups split
// the row's cells, each step they add their partial gradient sums through LDS
// in group order, and every group applies the same update to its register
// copy of the row (Eq. 5 with the step option and the clip).  The row starts
// at zero and is stored once, after the last step.  The per-cell work is the
// item pass's (process_block), so a step is the same computation as one
// launch of the item pass on the chunk.
// Stream records per lane per block in the extension kernel: a group's share
// of a free row of up to G * TSID_EXT_SPL cells stays in registers.
#ifndef TSID_EXT_SPL
#define TSID_EXT_SPL 4
#endif

template <int K, int V, bool BUF>
__global__ __launch_bounds__(kThreads) void k_extend_steps(const PassArgs A, int32_t steps) {
    constexpr int G = K / V;
    constexpr int NG = 64 / G;
    constexpr int SPL = (G * TSID_EXT_SPL) % chunk_cells<G>() == 0 ? TSID_EXT_SPL : chunk_cells<G>() / G;
    constexpr int SB = G * SPL;
    const int lane = threadIdx.x & 63;
    const int grp = lane / G, lg = lane % G, wv = threadIdx.x >> 6;
    const int64_t row = (int64_t)blockIdx.x * kWaves + wv;
    if (row >= A.rows) return;  // whole waves leave together
    const int64_t rb = A.ptr[row], deg = A.ptr[row + 1] - rb;
    if (A.skip_from > 0 && deg >= A.skip_from) return;  // the Gram-form kernel's row
    const int64_t beg = rb + grp * deg / NG, end = rb + (grp + 1) * deg / NG;
    const int64_t last = end - 1;
    const float s = A.degree ? 1.0f / (float)(deg > 1 ? deg : 1) : 1.0f;
    const YTable Yt = make_ytable<BUF>(A, K * 4);
    __shared__ float red[kWaves][NG][K];
    float x[V];
#pragma unroll
    for (int v = 0; v < V; ++v) x[v] = 0.f;
    const uint32_t xp[V / 2] = {};  // bf16 pairs: unused in fp32
    bool bad = false;
    // A group whose share of the row fits one stream block keeps its records
    // in registers for all steps (extension rows are short); longer shares
    // stream their records again each step.
    const bool one_block = end - beg <= SB;
    int2 keep[SPL], bufA[SPL], bufB[SPL];
    if (end > beg) {
#pragma unroll
        for (int c = 0; c < SPL; ++c) {
            const int64_t jj = beg + c * G + lg;
            keep[c] = load_cell(A.stream + (jj < last ? jj : last));
        }
    }
    // The row's gradient sum (the groups' partial sums in group order) and
    // the update of every group's copy of the row.
    auto update = [&](const float (&acc)[V]) {
        store_f32<V>(&red[wv][grp][lg * V], acc);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        float tot[V];
        load_f32<V>(&red[wv][0][lg * V], tot);
        for (int g = 1; g < NG; ++g) {
            float part[V];
            load_f32<V>(&red[wv][g][lg * V], part);
#pragma unroll
            for (int v = 0; v < V; ++v) tot[v] += part[v];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();  // every lane has read red before the next step writes it
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const float g = 2.0f * A.lam * x[v] - 2.0f * tot[v];
            const float d = clipped_step(g, s, A.clip, A.xi);
            x[v] = x[v] + A.lr * d;
            bad |= !__builtin_isfinite(x[v]);
        }
    };
    constexpr int CH = chunk_cells<G>();
    static_assert(CH <= SB && CH % G == 0, "a chunk lies inside the first stream block");
    if (deg <= (int64_t)NG * CH) {
        // Every group's share fits one chunk (shares differ by at most one
        // cell; the test is on the row, so the whole wave takes this branch):
        // the fixed rows are gathered once, into registers, and every step
        // reuses them, with the per-cell code's arithmetic in its order.
        float yc[CH][V], rc[CH];
        const int64_t left = end - beg;
        if (end > beg) {
#pragma unroll
            for (int t = 0; t < CH; ++t) {
                const int b = group_bcast<G>(keep[t / G].x, t % G);
                rc[t] = __int_as_float(group_bcast<G>(keep[t / G].y, t % G));
#pragma unroll
                for (int c = 0; c < V / 4; ++c) {
                    const uint4 q = ygather16<BUF>(Yt, b, K * 4, Lanes<G, V, false>::coord(lg, c) * 4);
                    yc[t][4 * c + 0] = __uint_as_float(q.x);
                    yc[t][4 * c + 1] = __uint_as_float(q.y);
                    yc[t][4 * c + 2] = __uint_as_float(q.z);
                    yc[t][4 * c + 3] = __uint_as_float(q.w);
                }
            }
        }
        for (int st = 0; st < steps; ++st) {
            float acc[V];
#pragma unroll
            for (int v = 0; v < V; ++v) acc[v] = 0.f;
            if (end > beg) {
#pragma unroll
                for (int t = 0; t < CH; ++t) {
                    float d = 0.f;
#pragma unroll
                    for (int v = 0; v < V; ++v) d += x[v] * yc[t][v];
                    d = group_sum<G>(d);
                    const float e = t < left ? rc[t] - d : 0.f;
#pragma unroll
                    for (int v = 0; v < V; ++v) acc[v] += e * yc[t][v];
                }
            }
            update(acc);
        }
    } else {
        for (int st = 0; st < steps; ++st) {
            float acc[V];
#pragma unroll
            for (int v = 0; v < V; ++v) acc[v] = 0.f;
            float e2 = 0.f;
            if (one_block) {
                if (end > beg)
                    process_block<K, V, false, false, BUF, false, SPL>(A, Yt, beg, end, last, lg, keep, bufB, x,
                                                                       xp, acc, e2);
            } else {
#pragma unroll
                for (int c = 0; c < SPL; ++c) bufA[c] = keep[c];
                for (int64_t j0 = beg; j0 < end; j0 += SB) {
                    process_block<K, V, false, false, BUF, true, SPL>(A, Yt, j0, end, last, lg, bufA, bufB, x, xp,
                                                                      acc, e2);
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int c = 0; c < SPL; ++c) bufA[c] = bufB[c];
                }
            }
            update(acc);
        }
    }
    if (grp == 0) store_coords<G, V, false>(A.Xn + row * K, lg, x);
    if (bad) A.err[ERR_NONFINITE] = 1;
}

template <int K>
__global__ void k_row_norms(const float *X, int32_t rows, float *norm) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= rows) return;
    float x[K];
    load_f32<K>(X + r * K, x);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < K; ++c) s += x[c] * x[c];
    norm[r] = s;
}

__global__ void k_to_bf16(const float *X, int64_t n, uint16_t *Xb) {
    for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n;
         j += (int64_t)gridDim.x * blockDim.x)
        Xb[j] = (uint16_t)bf16_bits(X[j]);
}

constexpr int kRedBlocks = 64;

// Four sums per slot: a (stride sa), b, c and d (strides nb, nc, nd); a null
// array sums to zero.
constexpr int kRedTerms = 4;
__global__ __launch_bounds__(256) void k_reduce_partial(const float *a, int64_t sa, int64_t na,
                                                        const float *b, int64_t nb, const float *c,
                                                        int64_t nc, const float *dd, int64_t nd,
                                                        double *partial) {
    __shared__ double lds[256];
    const int slot = blockIdx.y;
    const int which = blockIdx.x / kRedBlocks, blk = blockIdx.x % kRedBlocks;
    const float *src = which == 0   ? (a ? a + slot * sa : nullptr)
                       : which == 1 ? (b ? b + slot * nb : nullptr)
                       : which == 2 ? (c ? c + slot * nc : nullptr)
                                    : (dd ? dd + slot * nd : nullptr);
    const int64_t n = which == 0 ? na : (which == 1 ? nb : (which == 2 ? nc : nd));
    const int64_t chunk = (n + kRedBlocks - 1) / kRedBlocks;
    const int64_t lo = blk * chunk, hi = lo + chunk < n ? lo + chunk : n;
    double s = 0.0;
    if (src)
        for (int64_t j = lo + threadIdx.x; j < hi; j += 256) s += (double)src[j];
    lds[threadIdx.x] = s;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (threadIdx.x < off) lds[threadIdx.x] += lds[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) partial[(int64_t)slot * kRedTerms * kRedBlocks + blockIdx.x] = lds[0];
}

__global__ void k_reduce_final(const double *partial, int n_slots, double lam, double w4, double *out,
                               const int32_t *err, int32_t epoch0) {
    for (int slot = threadIdx.x; slot < n_slots; slot += blockDim.x) {
        if (err && epoch0 >= 0) {
            const int32_t f = err[ERR_NONFINITE];
            if (f != 0 && f - 1 < epoch0 + slot) continue;
        }
        const double *p = partial + (int64_t)slot * kRedTerms * kRedBlocks;
        double s[kRedTerms] = {0.0, 0.0, 0.0, 0.0};
        const int terms = w4 != 0.0 ? kRedTerms : kRedTerms - 1;  // the fourth only when weighted
        for (int w = 0; w < terms; ++w)
            for (int b = 0; b < kRedBlocks; ++b) s[w] += p[w * kRedBlocks + b];
        out[slot] = s[0] + lam * (s[1] + s[2]);
        if (w4 != 0.0) out[slot] += w4 * s[3];
    }
}

template <int K, int V, bool BF16>
void item_pass_kv(bool loss_only, const PassArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    constexpr int NG = 64 / (K / V);
    const int grid = ceil_div(a.n_items, (int64_t)kWaves * NG);
    if (grid <= 0) return;
    // buffer-resource gathers need the table (and every offset) below 2^31 bytes
    const bool buf = a.y_rows * (int64_t)K * (BF16 ? 2 : 4) < (int64_t(1) << 31);
    auto go = [&](auto kernel) {
        hipExtLaunchKernelGGL(kernel, dim3(grid), dim3(kThreads), 0, s, ev0, ev1, 0, a);
    };
    if (loss_only) {
        if (buf) go(k_item_pass<K, V, BF16, true, true>);
        else go(k_item_pass<K, V, BF16, true, false>);
    } else if (a.clip == 2) {
        if (buf) go(k_item_pass<K, V, BF16, false, true, true>);
        else go(k_item_pass<K, V, BF16, false, false, true>);
    } else {
        if (buf) go(k_item_pass<K, V, BF16, false, true>);
        else go(k_item_pass<K, V, BF16, false, false>);
    }
    TSID_HIP(hipGetLastError());
}

template <int K, int V, bool BF16>
void item_pass_sched_kv(const PassArgs &a, const int32_t *sched, int64_t n_wg, hipStream_t s, hipEvent_t ev0,
                        hipEvent_t ev1) {
    if (n_wg <= 0) return;
    if (n_wg > INT32_MAX) fail(TSID_E_INVAL, "too many workgroups");
    const bool buf = a.y_rows * (int64_t)K * (BF16 ? 2 : 4) < (int64_t(1) << 31);
    auto go = [&](auto kernel) {
        hipExtLaunchKernelGGL(kernel, dim3((unsigned)n_wg), dim3(kThreads), 0, s, ev0, ev1, 0, a, sched);
    };
    if (a.clip == 2) {
        if (buf) go(k_item_pass_sched<K, V, BF16, true, true>);
        else go(k_item_pass_sched<K, V, BF16, false, true>);
    } else {
        if (buf) go(k_item_pass_sched<K, V, BF16, true, false>);
        else go(k_item_pass_sched<K, V, BF16, false, false>);
    }
    TSID_HIP(hipGetLastError());
}

// Both sides' passes in one launch when their gathers use the same addressing;
// else two launches (ev0 on the first, ev1 on the second).
template <int K, int V, bool BF16>
void item_pass_pair_kv(const PassArgs &a0, const PassArgs &a1, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    constexpr int NG = 64 / (K / V);
    const int64_t g0 = ceil_div(a0.n_items, (int64_t)kWaves * NG), g1 = ceil_div(a1.n_items, (int64_t)kWaves * NG);
    const int64_t elt = BF16 ? 2 : 4;
    const bool buf0 = a0.y_rows * (int64_t)K * elt < (int64_t(1) << 31);
    const bool buf1 = a1.y_rows * (int64_t)K * elt < (int64_t(1) << 31);
    if (g0 <= 0 || g1 <= 0 || buf0 != buf1 || a0.clip != a1.clip || g0 + g1 > INT32_MAX) {
        item_pass_kv<K, V, BF16>(false, a0, s, ev0, nullptr);
        item_pass_kv<K, V, BF16>(false, a1, s, nullptr, ev1);
        return;
    }
    auto go = [&](auto kernel) {
        hipExtLaunchKernelGGL(kernel, dim3((unsigned)(g0 + g1)), dim3(kThreads), 0, s, ev0, ev1, 0, a0, a1,
                              (int32_t)g0);
    };
    if (a0.clip == 2) {
        if (buf0) go(k_item_pass_pair<K, V, BF16, true, true>);
        else go(k_item_pass_pair<K, V, BF16, false, true>);
    } else {
        if (buf0) go(k_item_pass_pair<K, V, BF16, true, false>);
        else go(k_item_pass_pair<K, V, BF16, false, false>);
    }
    TSID_HIP(hipGetLastError());
}

template <int K, int V, bool BF16>
void extend_steps_kv(const PassArgs &a, int32_t steps, hipStream_t s) {
    if constexpr (BF16) {
        fail(TSID_E_INVAL, "the extension runs in fp32");
    } else {
        const int grid = ceil_div(a.rows, (int64_t)kWaves);
        if (grid <= 0) return;  // steps == 0 still runs: it stores the zero start
        const bool buf = a.y_rows * (int64_t)K * 4 < (int64_t(1) << 31);
        if (buf)
            hipLaunchKernelGGL((k_extend_steps<K, V, true>), dim3(grid), dim3(kThreads), 0, s, a, steps);
        else
            hipLaunchKernelGGL((k_extend_steps<K, V, false>), dim3(grid), dim3(kThreads), 0, s, a, steps);
        TSID_HIP(hipGetLastError());
    }
}

template <int K, int V, bool BF16>
void block_combine_kv(const PassArgs &a, const float *part, int32_t n_blocks, hipStream_t s, hipEvent_t ev0,
                      hipEvent_t ev1) {
    constexpr int NG = 64 / (K / V);
    const int grid = ceil_div(a.rows, (int64_t)kWaves * NG);
    if (grid <= 0) return;
    hipExtLaunchKernelGGL(k_block_combine<K, V, BF16>, dim3(grid), dim3(kThreads), 0, s, ev0, ev1, 0, a, part,
                          n_blocks);
    TSID_HIP(hipGetLastError());
}

template <int K, int V, bool BF16>
void fixup_kv(const PassArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    constexpr int NG = 64 / (K / V);
    const int grid = ceil_div(a.rows, (int64_t)kWaves * NG);
    if (grid <= 0) return;
    hipExtLaunchKernelGGL(k_fixup<K, V, BF16>, dim3(grid), dim3(kThreads), 0, s, ev0, ev1, 0, a);
    TSID_HIP(hipGetLastError());
}

}  // namespace

// Coordinates per lane (V) for each rank: a cell is handled by G = K / V
// lanes.  Smaller G means fewer DPP and swizzle steps per cell; larger G means
// fewer distinct rows per gather instruction.
#ifndef TSID_V_F32_8
#define TSID_V_F32_8 4
#endif
#ifndef TSID_V_F32_16
#define TSID_V_F32_16 4
#endif
#ifndef TSID_V_F32_32
#define TSID_V_F32_32 4
#endif
#ifndef TSID_V_F32_64
#define TSID_V_F32_64 4
#endif
#ifndef TSID_V_F32_128
#define TSID_V_F32_128 8
#endif
#ifndef TSID_V_BF16_64
#define TSID_V_BF16_64 8
#endif
#ifndef TSID_V_BF16_128
#define TSID_V_BF16_128 16
#endif
#define TSID_DISPATCH_K(K_, FN, ...)                                                              \
    switch (K_) {                                                                                 \
        case 8: prec ? FN<8, 8, true>(__VA_ARGS__) : FN<8, TSID_V_F32_8, false>(__VA_ARGS__); break; \
        case 16: prec ? FN<16, 8, true>(__VA_ARGS__) : FN<16, TSID_V_F32_16, false>(__VA_ARGS__); break; \
        case 32: prec ? FN<32, 8, true>(__VA_ARGS__) : FN<32, TSID_V_F32_32, false>(__VA_ARGS__); break; \
        case 64: prec ? FN<64, TSID_V_BF16_64, true>(__VA_ARGS__)                                   \
                      : FN<64, TSID_V_F32_64, false>(__VA_ARGS__); break;                        \
        case 128: prec ? FN<128, TSID_V_BF16_128, true>(__VA_ARGS__)                                \
                       : FN<128, TSID_V_F32_128, false>(__VA_ARGS__); break;                     \
        default: fail(TSID_E_INVAL, "unsupported rank");                                         \
    }

void launch_item_pass(int K, int prec, bool loss_only, const PassArgs &a, hipStream_t s,
                      hipEvent_t ev0, hipEvent_t ev1) {
    TSID_DISPATCH_K(K, item_pass_kv, loss_only, a, s, ev0, ev1)
}

void launch_item_pass_pair(int K, int prec, const PassArgs &a0, const PassArgs &a1, hipStream_t s, hipEvent_t ev0,
                           hipEvent_t ev1) {
    TSID_DISPATCH_K(K, item_pass_pair_kv, a0, a1, s, ev0, ev1)
}

void launch_fixup(int K, int prec, const PassArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    TSID_DISPATCH_K(K, fixup_kv, a, s, ev0, ev1)
}

void launch_block_combine(int K, int prec, const PassArgs &a, const float *part, int32_t n_blocks, hipStream_t s,
                          hipEvent_t ev0, hipEvent_t ev1) {
    TSID_DISPATCH_K(K, block_combine_kv, a, part, n_blocks, s, ev0, ev1)
}

void launch_block_bounds(const int2 *stream, const int64_t *ptr, int32_t rows, int32_t n_blocks,
                         const int64_t *row_bounds, int64_t *bounds, hipStream_t s) {
    const int64_t n = (int64_t)(n_blocks + 1) * rows;
    if (n <= 0) return;
    k_block_bounds<<<ceil_div(n, 256), 256, 0, s>>>(stream, ptr, rows, n_blocks, row_bounds, bounds);
    TSID_HIP(hipGetLastError());
}

void launch_item_pass_sched(int K, int prec, const PassArgs &a, const int32_t *sched, int64_t n_wg, hipStream_t s,
                            hipEvent_t ev0, hipEvent_t ev1) {
    TSID_DISPATCH_K(K, item_pass_sched_kv, a, sched, n_wg, s, ev0, ev1)
}

void launch_extend_steps(int K, const PassArgs &a, int32_t steps, hipStream_t s) {
    const int prec = TSID_FP32;
    TSID_DISPATCH_K(K, extend_steps_kv, a, steps, s)
}

namespace {
template <int K, int V, bool BF16>
void groups_per_wave_kv(int &out) { out = 64 / (K / V); }
}  // namespace

int items_per_wave(int K, int prec) {
    int out = 0;
    TSID_DISPATCH_K(K, groups_per_wave_kv, out)
    return out;
}

int items_per_workgroup(int K, int prec) { return kWaves * items_per_wave(K, prec); }

void launch_row_norms(int K, const float *X, int32_t rows, float *norm, hipStream_t s) {
    if (rows <= 0) return;
    const int grid = ceil_div(rows, 256);
    switch (K) {
        case 8: k_row_norms<8><<<grid, 256, 0, s>>>(X, rows, norm); break;
        case 16: k_row_norms<16><<<grid, 256, 0, s>>>(X, rows, norm); break;
        case 32: k_row_norms<32><<<grid, 256, 0, s>>>(X, rows, norm); break;
        case 64: k_row_norms<64><<<grid, 256, 0, s>>>(X, rows, norm); break;
        case 128: k_row_norms<128><<<grid, 256, 0, s>>>(X, rows, norm); break;
        default: fail(TSID_E_INVAL, "unsupported rank");
    }
    TSID_HIP(hipGetLastError());
}

void launch_to_bf16(const float *X, int64_t n, uint16_t *Xb, hipStream_t s) {
    if (n <= 0) return;
    int64_t g = (n + 255) / 256;
    k_to_bf16<<<(int)(g > 65536 ? 65536 : g), 256, 0, s>>>(X, n, Xb);
    TSID_HIP(hipGetLastError());
}

size_t reduce_scratch_elems(int n_slots) { return (size_t)kRedTerms * kRedBlocks * (n_slots > 0 ? n_slots : 1); }

void launch_loss_reduce(const float *e2, int64_t e2_stride, int64_t ne, const float *np, int64_t nnp,
                        const float *nq, int64_t nnq, double lam, int n_slots, double *partial,
                        double *out, const int32_t *err, int32_t epoch0, hipStream_t s,
                        hipEvent_t ev0, hipEvent_t ev1, const float *ns, int64_t nns, double w4) {
    if (n_slots <= 0) return;
    if (!ns) w4 = 0.0;
    const int terms = w4 != 0.0 ? kRedTerms : kRedTerms - 1;
    hipExtLaunchKernelGGL(k_reduce_partial, dim3(terms * kRedBlocks, n_slots), dim3(256), 0, s, ev0,
                          nullptr, 0, e2, e2_stride, ne, np, nnp, nq, nnq, ns, nns, partial);
    TSID_HIP(hipGetLastError());
    hipExtLaunchKernelGGL(k_reduce_final, dim3(1), dim3(64), 0, s, nullptr, ev1, 0,
                          (const double *)partial, n_slots, lam, w4, out, err, epoch0);
    TSID_HIP(hipGetLastError());
}

}  // namespace tsid
