// Slab pass of the template fit (Stage I, Section 5.1) for templates whose
// observed cells are spread evenly over the template (uniform sampling, as in
// the scientific-data workloads).  Per observed cell it computes the residual
// e = r - p_a . q_b, aggregates the per-cell gradients of Eqs. 3-4 into the
// owning factor row and applies the row update of Eq. 5 (with the clip of
// Section 5.3), exactly as the item pass does; only the mapping differs.
//
// Mapping (gfx950, wave64, workgroups of kSlabLanes = 512 lanes, one per
// compute unit):
//  * One lane owns one factor row: a block of 512 consecutive owner rows per
//    workgroup.  The lane keeps the row and its gradient sum in registers for
//    the whole pass, so a cell costs k fused multiply-adds for the dot
//    product and k for the gradient, with no cross-lane reduction.
//  * The gathered factor is cut into slabs of C rows (128 KiB each).  The
//    workgroup copies one slab at a time into LDS with coalesced loads, then
//    every lane walks the cells of its row whose other index lies in the slab
//    (a run of the pass's own copy of the stream: 2 bytes of row within the
//    slab and 4 bytes of value per cell in 48-byte blocks of eight cells,
//    runs padded to whole blocks and stored slab-major; see SlabArgs) and
//    reads the other
//    factor rows from LDS.  A slab row is read
//    by every owner row of the block that observes it, so the gathers leave
//    the cache hierarchy and cost LDS bandwidth only.  A wave runs as long as
//    its busiest lane, so slabs are as large as LDS allows: the longer each
//    lane's run per slab, the smaller the relative spread between lanes.
//  * Lanes read the 16-byte chunks of an LDS row in an order rotated by their
//    lane id, so eight consecutive lanes touch eight different bank groups
//    whatever rows they read; the owner row and the gradient sum are held in
//    the same rotated order, which costs nothing.  gfx950 serves 16 lanes at
//    a time over 64 banks, and a 128-byte row sits in one half of them by the
//    parity of its index, so lanes x and x + 8 (same chunk index) would still
//    collide whenever their rows' parities agree: the pass walks its own copy
//    of the stream in which each run lists the cells of one parity first --
//    even for lanes with bit 3 clear, odd for the others (k_slab_order).
//  * A workgroup covers a range of S slabs.  When a block of rows is split
//    over several workgroups (U > 1) each leaves its partial gradient sums in
//    a carry buffer, and a second kernel adds the U parts of every row in a
//    fixed order and updates the row.  No atomic operation is used, and the
//    result does not depend on the order in which workgroups run.
#include <hip/hip_ext.h>

#include "internal.h"

namespace tsid {

namespace {

constexpr int kLanes = kSlabLanes;

// Waves per SIMD the register budget must allow (one 512-lane workgroup per
// compute unit: two).
#ifndef TSID_SLAB_WAVES_PER_EU
#define TSID_SLAB_WAVES_PER_EU 2
#endif
// Dependency chains of the dot product (1: one chain of k fused multiply-adds).
#ifndef TSID_SLAB_CHAINS
#define TSID_SLAB_CHAINS 4
#endif

__device__ __forceinline__ float4 f4_zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }

// Chunk of the row held in register slot c of this lane (rotation by lane id;
// NCH is a power of two).
template <int NCH>
__device__ __forceinline__ int slot_chunk(int c, int rot) {
    return (c + rot) & (NCH - 1);
}

// Eq. 5 (descent on the summed gradients of Eqs. 3-4), the 1/max(1, deg)
// normalisation of the degree step and the Section 5.3 clip, for one row held
// by one lane in rotated chunk order.
template <int K>
__device__ __forceinline__ void finalize_lane(const SlabArgs &A, int xr, int rot,
                                              const float4 (&x)[K / 4], const float4 (&acc)[K / 4]) {
    constexpr int NCH = K / 4;
    const int64_t deg = A.ptr[xr + 1] - A.ptr[xr];
    const float s = A.degree ? 1.0f / (float)(deg > 1 ? deg : 1) : 1.0f;
    float4 *out = reinterpret_cast<float4 *>(A.Xn + (int64_t)xr * K);
    bool bad = false;
    float nrm = 0.f;
    auto upd = [&](float xv, float av) {
        const float g = 2.0f * A.lam * xv - 2.0f * av;
        const float d = clipped_step(g, s, A.clip, A.xi);
        const float xn = xv + A.lr * d;
        bad |= !__builtin_isfinite(xn);
        nrm += xv * xv;
        return xn;
    };
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        float4 o;
        o.x = upd(x[c].x, acc[c].x);
        o.y = upd(x[c].y, acc[c].y);
        o.z = upd(x[c].z, acc[c].z);
        o.w = upd(x[c].w, acc[c].w);
        out[slot_chunk<NCH>(c, rot)] = o;
    }
    if (A.norm) A.norm[xr] = nrm;
    if (bad) A.err[ERR_NONFINITE] = A.epoch + 1;
}

// The eight records of a run from record j (a multiple of 8): one 48-byte
// block, their rows within the slab and their values.  A lane reads its run
// block after block, so it has one partly read 128-byte line at a time.
struct Burst {
    uint4 ix;        // eight 16-bit rows, two per word (low half first)
    float4 v0, v1;   // the eight values
};

__device__ __forceinline__ void load_burst(const SlabArgs &A, uint32_t j, Burst &b) {
    const uint4 *blk = A.sblk + (size_t)(j >> 3) * 3;
    b.ix = blk[0];
    b.v0 = __builtin_bit_cast(float4, blk[1]);
    b.v1 = __builtin_bit_cast(float4, blk[2]);
}

// First record of burst i of the run [p, q): forwards, or backwards from its
// end.
__device__ __forceinline__ uint32_t burst_at(uint32_t p, uint32_t q, int32_t i, bool back) {
    return back ? q - 8u * (uint32_t)(i + 1) : p + 8u * (uint32_t)i;
}

template <int K>
__device__ __forceinline__ void slab_read_row(const char *ysb, uint32_t row_off, const uint32_t (&koff)[K / 4],
                                              float4 (&y)[K / 4]) {
#pragma unroll
    for (int i = 0; i < K / 4; ++i) y[i] = *reinterpret_cast<const float4 *>(ysb + row_off + koff[i]);
}

// One cell: residual against its LDS row, e^2 and the gradient sum.  A pad
// reads the zero row with value 0, so it adds exactly nothing.
template <int K, bool LOSS_ONLY>
__device__ __forceinline__ void slab_cell(const float4 (&y)[K / 4], float r, const float4 (&x)[K / 4],
                                          float4 (&acc)[K / 4], float &e2) {
    constexpr int NCH = K / 4;
#if TSID_SLAB_CHAINS == 1
    float d = 0.f;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        d += x[i].x * y[i].x;
        d += x[i].y * y[i].y;
        d += x[i].z * y[i].z;
        d += x[i].w * y[i].w;
    }
#else
    float d0 = 0.f, d1 = 0.f, d2 = 0.f, d3 = 0.f;
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
        d0 += x[i].x * y[i].x;
        d1 += x[i].y * y[i].y;
        d2 += x[i].z * y[i].z;
        d3 += x[i].w * y[i].w;
    }
    const float d = (d0 + d1) + (d2 + d3);
#endif
    const float e = r - d;
    e2 += e * e;
    if constexpr (!LOSS_ONLY) {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            acc[i].x += e * y[i].x;
            acc[i].y += e * y[i].y;
            acc[i].z += e * y[i].z;
            acc[i].w += e * y[i].w;
        }
    }
}

// The eight cells of a burst.  The LDS reads of cell c + 1 are issued before
// the arithmetic of cell c, so a wave has one row in flight while it
// computes.
template <int K, bool LOSS_ONLY>
__device__ __forceinline__ void slab_burst(const Burst &b, const char *ysb, const uint32_t (&koff)[K / 4],
                                           const float4 (&x)[K / 4], float4 (&acc)[K / 4], float &e2) {
    constexpr int NCH = K / 4;
    constexpr uint32_t RB = K * 4;  // bytes per LDS row
    const uint32_t w[4] = {b.ix.x, b.ix.y, b.ix.z, b.ix.w};
    uint32_t off[8];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        off[2 * c] = (w[c] & 0xffffu) * RB;
        off[2 * c + 1] = (w[c] >> 16) * RB;
    }
    const float r[8] = {b.v0.x, b.v0.y, b.v0.z, b.v0.w, b.v1.x, b.v1.y, b.v1.z, b.v1.w};
    if constexpr (K > 32) {
        // k = 64: two rows of 64 registers in flight would spill; read and
        // compute two cells at a time instead
#pragma unroll
        for (int c = 0; c < 8; c += 2) {
            __builtin_amdgcn_sched_barrier(0);
            float4 y0[NCH], y1[NCH];
            slab_read_row<K>(ysb, off[c], koff, y0);
            slab_read_row<K>(ysb, off[c + 1], koff, y1);
            slab_cell<K, LOSS_ONLY>(y0, r[c], x, acc, e2);
            slab_cell<K, LOSS_ONLY>(y1, r[c + 1], x, acc, e2);
        }
        return;
    }
    float4 ya[NCH], yb[NCH];
    slab_read_row<K>(ysb, off[0], koff, ya);
#pragma unroll
    for (int c = 0; c < 8; c += 2) {
        __builtin_amdgcn_sched_barrier(0);
        slab_read_row<K>(ysb, off[c + 1], koff, yb);
        slab_cell<K, LOSS_ONLY>(ya, r[c], x, acc, e2);
        __builtin_amdgcn_sched_barrier(0);
        if (c + 2 < 8) slab_read_row<K>(ysb, off[c + 2], koff, ya);
        slab_cell<K, LOSS_ONLY>(yb, r[c + 1], x, acc, e2);
    }
}

// Workgroup u of one side's pass.
template <int K, bool LOSS_ONLY>
__device__ __forceinline__ void slab_pass_unit(const SlabArgs &A, const int u) {
    constexpr int NCH = K / 4;                        // 16-byte chunks per factor row
    constexpr int RM = (NCH < 8 ? NCH : 8) - 1;       // lane rotation mask
    static_assert((NCH & (NCH - 1)) == 0, "rows hold a power-of-two number of chunks");
    extern __shared__ float4 ys[];                    // one slab (C rows x NCH chunks), then a zero row
    if (A.skip_after_nonfinite) {
        const int32_t f = A.err[ERR_NONFINITE];
        if (f != 0 && f - 1 < A.epoch) return;  // same outcome for every workgroup
    }
    const int tid = threadIdx.x;
    const int U = A.units_per_block;
    const int blk = u / U, ur = u - blk * U;
    const int s0 = ur * A.slabs_per_unit;
    const int s1 = min(s0 + A.slabs_per_unit, A.n_slabs);
    const int xr = blk * kLanes + tid;
    const bool own = xr < A.rows;
    const int rot = tid & RM;
    const bool back = (xr & 1) != 0;  // this row walks its runs backwards

    float4 x[NCH], acc[NCH];
    uint32_t koff[NCH];  // byte offset of slot c's chunk within an LDS row
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        koff[c] = (uint32_t)slot_chunk<NCH>(c, rot) * 16u;
        x[c] = own ? reinterpret_cast<const float4 *>(A.X + (int64_t)xr * K)[slot_chunk<NCH>(c, rot)]
                   : f4_zero();
        acc[c] = f4_zero();
    }
    float e2 = 0.f;

    const float4 *Y4 = reinterpret_cast<const float4 *>(A.Y);
    constexpr int nf4 = kSlabBytes / 16;              // chunks per slab
    static_assert(nf4 % kLanes == 0, "every lane copies the same number of chunks");
    const int64_t ylast = (int64_t)A.y_rows * NCH - 1;  // last chunk of the table
    const char *ysb = reinterpret_cast<const char *>(ys);
    constexpr int NF = nf4 / kLanes;  // slab chunks each lane copies
    // LDS byte address of this wave's first chunk in each copy round: the
    // direct global-to-LDS loads write 16 bytes per lane at consecutive
    // addresses from a wave-uniform base.
    const int wave_base = __builtin_amdgcn_readfirstlane(tid & ~63);
    // the row the pads read (the slab copies never write it; the first
    // barrier below orders this store before any read)
    if (tid < NCH) ys[nf4 + tid] = f4_zero();
    for (int s = s0; s < s1; ++s) {
        // The lane's run bounds and its first records are requested before
        // the barrier, the slab right after it with every copy in flight, so
        // the workgroup waits for about one memory round trip per slab.
        uint32_t p = 0, q = 0;
        if (own) {
            p = A.seg[(int64_t)s * A.rows + xr];
            q = A.seg[(int64_t)s * A.rows + xr + 1];
        }
        Burst ba, bc;
        if (p < q) load_burst(A, burst_at(p, q, 0, back), ba);
        __syncthreads();  // every lane is done with the previous slab
        // Chunks past the table's end (last slab only) repeat its last chunk;
        // no cell refers to those LDS rows.
        const int64_t g0 = (int64_t)s * nf4 + tid;
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const int64_t g = g0 + (int64_t)f * kLanes;
            __builtin_amdgcn_global_load_lds(Y4 + (g < ylast ? g : ylast),
                                             (__attribute__((address_space(3))) void *)(ys + f * kLanes + wave_base),
                                             16, 0, 0);
        }
        __builtin_amdgcn_s_waitcnt(0);  // the copies have landed in LDS
        __syncthreads();
        // The lane's cells in this slab (a whole number of bursts of eight
        // records); the next burst's records load while this one computes.
        // Odd rows walk their runs backwards: a line shared by the runs of
        // rows x and x + 1 (adjacent in memory) is then read by both lanes
        // at about the same time, at the start or at the end of their runs,
        // rather than once at each end of the slab.
        const int32_t n = (int32_t)(q - p) >> 3;
        for (int32_t i = 0; i < n; i += 2) {
            if (i + 1 < n) load_burst(A, burst_at(p, q, i + 1, back), bc);
            slab_burst<K, LOSS_ONLY>(ba, ysb, koff, x, acc, e2);
            if (i + 1 >= n) break;
            if (i + 2 < n) load_burst(A, burst_at(p, q, i + 2, back), ba);
            slab_burst<K, LOSS_ONLY>(bc, ysb, koff, x, acc, e2);
        }
    }

    if (A.e2) A.e2[(int64_t)u * kLanes + tid] = e2;
    if constexpr (LOSS_ONLY) {
        if (A.norm && own && ur == 0) {
            float nrm = 0.f;
#pragma unroll
            for (int c = 0; c < NCH; ++c)
                nrm += x[c].x * x[c].x + x[c].y * x[c].y + x[c].z * x[c].z + x[c].w * x[c].w;
            A.norm[xr] = nrm;
        }
    } else {
        if (U == 1) {
            if (own) finalize_lane<K>(A, xr, rot, x, acc);
            return;
        }
        // Partial sums of this unit (natural chunk order); k_slab_finish adds
        // the U parts of each row in unit order and updates the row.
        if (own) {
            float4 *cp = reinterpret_cast<float4 *>(A.carry + ((int64_t)u * kLanes + tid) * K);
#pragma unroll
            for (int c = 0; c < NCH; ++c) cp[slot_chunk<NCH>(c, rot)] = acc[c];
        }
    }
}

template <int K, bool LOSS_ONLY>
__global__ __launch_bounds__(kLanes) __attribute__((amdgpu_waves_per_eu(TSID_SLAB_WAVES_PER_EU)))
void k_slab_pass(const SlabArgs A) {
    slab_pass_unit<K, LOSS_ONLY>(A, blockIdx.x);
}

// Both passes of a simultaneous step in one launch: they read only the old
// factors and write disjoint outputs, so the n0 workgroups of the P pass
// (A0) and then those of the Q pass (A1) share one grid, and the Q pass's
// workgroups start as the P pass's leave the compute units instead of after
// the whole P pass has drained.
template <int K>
__global__ __launch_bounds__(kLanes) __attribute__((amdgpu_waves_per_eu(TSID_SLAB_WAVES_PER_EU)))
void k_slab_pass_pair(const SlabArgs A0, const SlabArgs A1, const int32_t n0) {
    const int u = blockIdx.x;
    if (u < n0)
        slab_pass_unit<K, false>(A0, u);
    else
        slab_pass_unit<K, false>(A1, u - n0);
}

// Blocks split over U > 1 workgroups: the U partial sums of every row are
// added in unit order, then the row takes the update of Eq. 5.  One lane per
// 16-byte chunk of a row (NCH consecutive lanes per row), so every load is
// coalesced and all U loads of a lane are in flight together.
// Thread t of one side's finish (whole workgroups of 256 take one side).
template <int K>
__device__ __forceinline__ void slab_finish_lane(const SlabArgs &A, const int64_t t) {
    constexpr int NCH = K / 4;
    static_assert(NCH <= 64 && (64 % NCH) == 0, "a row's lanes sit inside one wave");
    if (A.skip_after_nonfinite) {
        const int32_t f = A.err[ERR_NONFINITE];
        if (f != 0 && f - 1 < A.epoch) return;
    }
    const int64_t xr = t / NCH;
    const int ch = (int)(t % NCH);
    const bool own = xr < A.rows;
    const int64_t xs = own ? xr : 0;  // rows past the end mirror row 0 and store nothing
    const int U = A.units_per_block;
    const int64_t blk = xs / kLanes, lane = xs % kLanes;
    const float4 *cp = reinterpret_cast<const float4 *>(A.carry) + ((blk * U) * kLanes + lane) * NCH + ch;
    const int64_t unit_stride = (int64_t)kLanes * NCH;  // float4 between consecutive units
    float4 tot = f4_zero();
    int v = 0;
    for (; v + 4 <= U; v += 4) {
        float4 q[4];
#pragma unroll
        for (int w = 0; w < 4; ++w) q[w] = cp[(v + w) * unit_stride];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            tot.x += q[w].x;
            tot.y += q[w].y;
            tot.z += q[w].z;
            tot.w += q[w].w;
        }
    }
    for (; v < U; ++v) {
        const float4 q = cp[v * unit_stride];
        tot.x += q.x;
        tot.y += q.y;
        tot.z += q.z;
        tot.w += q.w;
    }
    const float4 x = reinterpret_cast<const float4 *>(A.X + xs * K)[ch];
    const int64_t deg = A.ptr[xs + 1] - A.ptr[xs];
    const float s = A.degree ? 1.0f / (float)(deg > 1 ? deg : 1) : 1.0f;
    bool bad = false;
    float nrm = 0.f;
    auto upd = [&](float xv, float av) {
        const float g = 2.0f * A.lam * xv - 2.0f * av;
        const float d = clipped_step(g, s, A.clip, A.xi);
        const float xn = xv + A.lr * d;
        bad |= !__builtin_isfinite(xn);
        nrm += xv * xv;
        return xn;
    };
    float4 o;
    o.x = upd(x.x, tot.x);
    o.y = upd(x.y, tot.y);
    o.z = upd(x.z, tot.z);
    o.w = upd(x.w, tot.w);
    // row norm over the NCH lanes of the row (butterfly: every lane ends with
    // the same bits)
#pragma unroll
    for (int off = 1; off < NCH; off <<= 1) nrm += __shfl_xor(nrm, off, 64);
    if (own) {
        reinterpret_cast<float4 *>(A.Xn + xr * K)[ch] = o;
        if (A.norm && ch == 0) A.norm[xr] = nrm;
        if (bad) A.err[ERR_NONFINITE] = A.epoch + 1;
    }
}

template <int K>
__global__ __launch_bounds__(256) void k_slab_finish(const SlabArgs A) {
    slab_finish_lane<K>(A, (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

// The finishes of both passes in one launch: workgroups below b0 take the P
// pass's rows, the rest the Q pass's.
template <int K>
__global__ __launch_bounds__(256) void k_slab_finish_pair(const SlabArgs A0, const SlabArgs A1, const int32_t b0) {
    const int b = blockIdx.x;
    if (b < b0)
        slab_finish_lane<K>(A0, (int64_t)b * 256 + threadIdx.x);
    else
        slab_finish_lane<K>(A1, (int64_t)(b - b0) * 256 + threadIdx.x);
}

// seg[s * rows + x] = first cell of bucket x whose other index is >= s * C
// (binary search in the bucket's sorted other indices), s = 0..n_slabs.
__global__ void k_slab_seg(const int2 *stream, const int64_t *ptr, int32_t rows, int32_t n_slabs,
                           int32_t C, uint32_t *seg) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)(n_slabs + 1) * rows) return;
    const int32_t s = (int32_t)(t / rows), x = (int32_t)(t % rows);
    const int64_t key = (int64_t)s * C;
    int64_t lo = ptr[x], hi = ptr[x + 1];
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if ((int64_t)stream[mid].x < key) lo = mid + 1;
        else hi = mid;
    }
    seg[t] = (uint32_t)lo;
}

// Slabs above 64 KiB need the kernel's dynamic LDS limit raised (once).
template <typename Kern>
void allow_lds(Kern kernel, size_t bytes) {
    if (bytes > 64 * 1024)
        TSID_HIP(hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes));
}

// The slab pass's own copy of a bucketed stream (see SlabArgs).  Within
// every run (x, s) the cells whose other index b has the parity
// (x >> 3) & 1 come first, then the rest, each part in the stream's order,
// then the pads.  A staged LDS row lies in one half of the 64 banks
// according to the parity of b, and the lanes x and x + 8 of a 16-lane LDS
// group read the same chunk index (lane rotation), so with this order they
// read opposite halves for most of their runs instead of colliding whenever
// their rows' parities agree.  Runs are stored slab-major, so the runs one
// workgroup walks in a slab are one contiguous stretch of memory, and a line
// shared by two runs is read by neighbouring lanes at the same time.
__global__ void k_slab_order(const int2 *stream, const uint32_t *seg, int32_t rows, int32_t n_slabs, int32_t C,
                             const uint32_t *pseg, uint4 *sblk) {
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n_slabs * rows) return;
    const int32_t s = (int32_t)(t / rows), x = (int32_t)(t % rows);
    const uint32_t p = seg[(int64_t)s * rows + x], q = seg[(int64_t)(s + 1) * rows + x];
    const int first = (x >> 3) & 1;
    const int32_t base = s * C;
    // record o: 16-bit row o % 8 of block o / 8, then value o % 8 after the
    // block's 16 bytes of rows
    uint16_t *const rows16 = reinterpret_cast<uint16_t *>(sblk);
    float *const vals = reinterpret_cast<float *>(sblk);
    auto put = [&](uint32_t o, uint16_t r, float v) {
        const size_t g = (size_t)(o >> 3) * 24, i = o & 7;  // block start in 16-bit units
        rows16[g + i] = r;
        vals[g / 2 + 4 + i] = v;
    };
    uint32_t o = pseg[t];
    for (int pass = 0; pass < 2; ++pass) {
        for (uint32_t j = p; j < q; ++j) {
            const int2 c = stream[j];
            if (((c.x & 1) == first) == (pass == 0)) put(o++, (uint16_t)(c.x - base), __int_as_float(c.y));
        }
    }
    for (const uint32_t e = pseg[t + 1]; o < e; ++o) put(o, (uint16_t)C, 0.f);
}

template <int K>
void slab_pass_k(bool loss_only, const SlabArgs &a, int64_t n_units, hipStream_t s, hipEvent_t ev0,
                 hipEvent_t ev1) {
    const size_t lds = (size_t)(a.C + 1) * K * 4;  // the slab and the zero row
    static const bool lds_ok = (allow_lds(k_slab_pass<K, true>, kSlabBytes + K * 4),
                                allow_lds(k_slab_pass<K, false>, kSlabBytes + K * 4), true);
    (void)lds_ok;
    if (loss_only)
        hipExtLaunchKernelGGL(k_slab_pass<K, true>, dim3((unsigned)n_units), dim3(kLanes), lds, s, ev0, ev1,
                              0, a);
    else
        hipExtLaunchKernelGGL(k_slab_pass<K, false>, dim3((unsigned)n_units), dim3(kLanes), lds, s, ev0,
                              ev1, 0, a);
    TSID_HIP(hipGetLastError());
}

template <int K>
void slab_finish_k(const SlabArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    const int64_t threads = (int64_t)a.rows * (K / 4);
    const unsigned blocks = (unsigned)((threads + 255) / 256);
    hipExtLaunchKernelGGL(k_slab_finish<K>, dim3(blocks), dim3(256), 0, s, ev0, ev1, 0, a);
    TSID_HIP(hipGetLastError());
}

template <int K>
void slab_pass_pair_k(const SlabArgs &a0, int64_t n0, const SlabArgs &a1, int64_t n1, hipStream_t s,
                      hipEvent_t ev0, hipEvent_t ev1) {
    const size_t lds = (size_t)(a0.C + 1) * K * 4;
    static const bool lds_ok = (allow_lds(k_slab_pass_pair<K>, kSlabBytes + K * 4), true);
    (void)lds_ok;
    hipExtLaunchKernelGGL(k_slab_pass_pair<K>, dim3((unsigned)(n0 + n1)), dim3(kLanes), lds, s, ev0, ev1, 0, a0,
                          a1, (int32_t)n0);
    TSID_HIP(hipGetLastError());
}

template <int K>
void slab_finish_pair_k(const SlabArgs &a0, const SlabArgs &a1, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    const int64_t b0 = ((int64_t)a0.rows * (K / 4) + 255) / 256, b1 = ((int64_t)a1.rows * (K / 4) + 255) / 256;
    hipExtLaunchKernelGGL(k_slab_finish_pair<K>, dim3((unsigned)(b0 + b1)), dim3(256), 0, s, ev0, ev1, 0, a0, a1,
                          (int32_t)b0);
    TSID_HIP(hipGetLastError());
}

}  // namespace

bool slab_supported(int K, int prec) {
    return prec == TSID_FP32 && (K == 8 || K == 16 || K == 32 || K == 64);
}

int slab_rows(int K) { return kSlabBytes / (4 * K); }

void launch_slab_seg(const int2 *stream, const int64_t *ptr, int32_t rows, int32_t n_slabs, int32_t C,
                     uint32_t *seg, hipStream_t s) {
    const int64_t n = (int64_t)(n_slabs + 1) * rows;
    if (n <= 0) return;
    k_slab_seg<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(stream, ptr, rows, n_slabs, C, seg);
    TSID_HIP(hipGetLastError());
}

void launch_slab_order(const int2 *stream, const uint32_t *seg, int32_t rows, int32_t n_slabs, int32_t C,
                       const uint32_t *pseg, uint4 *sblk, hipStream_t s) {
    const int64_t n = (int64_t)n_slabs * rows;
    if (n <= 0) return;
    k_slab_order<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(stream, seg, rows, n_slabs, C, pseg, sblk);
    TSID_HIP(hipGetLastError());
}

void launch_slab_finish(int K, const SlabArgs &a, hipStream_t s, hipEvent_t ev0, hipEvent_t ev1) {
    if (a.rows <= 0) return;
    switch (K) {
        case 8: slab_finish_k<8>(a, s, ev0, ev1); break;
        case 16: slab_finish_k<16>(a, s, ev0, ev1); break;
        case 32: slab_finish_k<32>(a, s, ev0, ev1); break;
        case 64: slab_finish_k<64>(a, s, ev0, ev1); break;
        default: fail(TSID_E_INVAL, "the slab pass supports k = 8, 16, 32, 64");
    }
}

void launch_slab_pass_pair(int K, const SlabArgs &a0, int64_t n0, const SlabArgs &a1, int64_t n1, hipStream_t s,
                           hipEvent_t ev0, hipEvent_t ev1) {
    if (n0 <= 0 || n1 <= 0 || a0.C != a1.C || n0 + n1 > INT32_MAX)
        fail(TSID_E_INVAL, "paired slab passes need workgroups on both sides and one slab size");
    switch (K) {
        case 8: slab_pass_pair_k<8>(a0, n0, a1, n1, s, ev0, ev1); break;
        case 16: slab_pass_pair_k<16>(a0, n0, a1, n1, s, ev0, ev1); break;
        case 32: slab_pass_pair_k<32>(a0, n0, a1, n1, s, ev0, ev1); break;
        case 64: slab_pass_pair_k<64>(a0, n0, a1, n1, s, ev0, ev1); break;
        default: fail(TSID_E_INVAL, "the slab pass supports k = 8, 16, 32, 64");
    }
}

void launch_slab_finish_pair(int K, const SlabArgs &a0, const SlabArgs &a1, hipStream_t s, hipEvent_t ev0,
                             hipEvent_t ev1) {
    if (a0.rows <= 0 || a1.rows <= 0) fail(TSID_E_INVAL, "paired slab finishes need rows on both sides");
    switch (K) {
        case 8: slab_finish_pair_k<8>(a0, a1, s, ev0, ev1); break;
        case 16: slab_finish_pair_k<16>(a0, a1, s, ev0, ev1); break;
        case 32: slab_finish_pair_k<32>(a0, a1, s, ev0, ev1); break;
        case 64: slab_finish_pair_k<64>(a0, a1, s, ev0, ev1); break;
        default: fail(TSID_E_INVAL, "the slab pass supports k = 8, 16, 32, 64");
    }
}

void launch_slab_pass(int K, bool loss_only, const SlabArgs &a, int64_t n_units, hipStream_t s,
                      hipEvent_t ev0, hipEvent_t ev1) {
    if (n_units <= 0) return;
    switch (K) {
        case 8: slab_pass_k<8>(loss_only, a, n_units, s, ev0, ev1); break;
        case 16: slab_pass_k<16>(loss_only, a, n_units, s, ev0, ev1); break;
        case 32: slab_pass_k<32>(loss_only, a, n_units, s, ev0, ev1); break;
        case 64: slab_pass_k<64>(loss_only, a, n_units, s, ev0, ev1); break;
        default: fail(TSID_E_INVAL, "the slab pass supports k = 8, 16, 32, 64");
    }
}

}  // namespace tsid
