// libtsid C ABI: context, argument validation, the template build, the
// epoch loop of the template fit, the loss, and the chunked extension
// pipeline.  See include/tsid.h for the contract of every entry point.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <unordered_map>
#include <utility>
#include <vector>

#include "internal.h"

namespace tsid {

void fail(tsid_status st, const std::string &msg) { throw Error{st, msg}; }

void hip_check(hipError_t e, const char *what) {
    if (e != hipSuccess) fail(TSID_E_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

namespace {

constexpr int64_t kDefaultStage = int64_t(1) << 24;  // entries per host-to-device piece
constexpr int64_t kMaxEntries = (int64_t(1) << 32) - 1;

bool valid_rank(int32_t k) { return k == 8 || k == 16 || k == 32 || k == 64 || k == 128; }

// Entries per work item: enough items to keep every compute unit busy, long
// enough that the per-item overhead (owner row load, final store) stays small.
#ifndef TSID_TARGET_ITEMS
#define TSID_TARGET_ITEMS 131072
#endif
// Work items of a mini-batch step: each batch holds a fraction of the cells
// but every owner row still costs its row load and update.
#ifndef TSID_MB_TARGET_ITEMS
#define TSID_MB_TARGET_ITEMS 131072
#endif
int32_t choose_E(int64_t nnz, int64_t target = TSID_TARGET_ITEMS) {
    int64_t e = (nnz + target - 1) / target;
    e = (e + 15) / 16 * 16;
    if (e < 64) e = 64;
    if (e > 4096) e = 4096;
    return (int32_t)e;
}

}  // namespace

// Device memory owned by a context, with an optional byte cap.
struct Arena {
    size_t cap = 0, used = 0;
    std::unordered_map<void *, size_t> sizes;

    template <typename T>
    T *alloc(int64_t count) {
        size_t bytes = (size_t)(count > 0 ? count : 1) * sizeof(T);
        bytes = (bytes + 255) & ~size_t(255);
        if (cap && used + bytes > cap) fail(TSID_E_NOMEM, "device byte cap exceeded");
        void *p = nullptr;
        if (hipMalloc(&p, bytes) != hipSuccess) {
            (void)hipGetLastError();
            fail(TSID_E_NOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
        }
        sizes[p] = bytes;
        used += bytes;
        return static_cast<T *>(p);
    }
    template <typename T>
    void release(T *&p) {
        if (!p) return;
        auto it = sizes.find((void *)p);
        if (it != sizes.end()) {
            used -= it->second;
            sizes.erase(it);
        }
        (void)hipFree((void *)p);
        p = nullptr;
    }
};

// Work plan of one pass for one precision (the lane grouping, hence the
// groups per wave, depends on it).
struct Plan {
    bool ready = false;
    uint32_t *item_off = nullptr;  // first item of each bucket
    uint32_t *item_end = nullptr;  // one past its last item
    int32_t *items = nullptr;      // bucket of each item, -1 for pads
    int32_t n_items = 0;
    int32_t E = 64;
    bool spans = true;             // some bucket's items span two waves (fixup needed)
};

// Slab pass of one side (fp32): slab pointers, the carry of partial sums and
// the unit split.  `use` says whether the fit runs this side's pass with
// the slab kernel.
struct SlabPlan {
    bool ready = false, use = false;
    int32_t suits = -1;        // cached slab_suits() of the template (-1: not evaluated)
    int32_t C = 0, n_slabs = 0, S = 0, U = 0, n_blocks = 0;
    uint32_t *seg = nullptr;   // run pointers of the pass's copy of the stream (SlabArgs)
    uint4 *sblk = nullptr;     // the copy itself (launch_slab_order)
    float *carry = nullptr;
    int64_t units() const { return (int64_t)n_blocks * U; }
    int64_t lanes() const { return units() * kSlabLanes; }
};

// Dense head tiles of a bf16 fit (dense.hip): for each side the stripe
// pointers, the other-side tile index and the owner-major values of every
// dense tile, the streams of the remaining (sparse) cells with their bucket
// pointers and work plans, and the per-row dense gradient sums.
struct DensePlan {
    bool ready = false;
    float fill = 0.f;          // tile fill it was built for
    int64_t tiles = 0, cells = 0, sparse_nnz = 0;
    int64_t stripes[2] = {0, 0};  // stripes holding a dense tile, per side
    uint32_t *tile_ptr[2] = {nullptr, nullptr};
    // work segments (one wave each) and the stripes split over several
    int64_t n_segs[2] = {0, 0}, n_multi[2] = {0, 0};
    uint32_t *seg_tile[2] = {nullptr, nullptr};
    int32_t *seg_order[2] = {nullptr, nullptr};  // launch order of the segments
    int32_t *seg_stripe[2] = {nullptr, nullptr};
    uint32_t *stripe_seg[2] = {nullptr, nullptr};
    int32_t *multi[2] = {nullptr, nullptr};
    float *part[2] = {nullptr, nullptr};
    int32_t *tile_other[2] = {nullptr, nullptr};
    float *R[2] = {nullptr, nullptr};
    int2 *sparse[2] = {nullptr, nullptr};
    int64_t *sparse_ptr[2] = {nullptr, nullptr};
    Plan plan[2];
    float *gd[2] = {nullptr, nullptr};
};

// Mini-batch epochs (minibatch.hip): batch-major copies of both streams,
// the bucket pointers of every batch (batch beta of side s: ptr[s] +
// beta * rows, rows + 1 entries) and, per precision, every batch's work plan.
struct MiniPlan {
    bool ready = false;
    int32_t B = 0;
    uint64_t seed = 0;
    int2 *stream[2] = {nullptr, nullptr};
    int64_t *ptr[2] = {nullptr, nullptr};
    std::vector<int64_t> hptr[2];     // host copies (B * rows + 1)
    std::vector<Plan> plan[2][2];     // [side][precision], B plans once built
    int64_t max_items[2] = {0, 0};    // [precision]: largest plan
};

// Multi-view similarity term (similarity.hip): S over the template's
// columns as CSR, its weight, the per-column gradient sums and a ring of
// per-column loss terms (one slot per epoch of the loss ring).
struct SimPlan {
    bool on = false;
    float beta = 0.f;
    int64_t nnz = 0;
    int64_t *ptr = nullptr;
    int32_t *col = nullptr;
    float *val = nullptr;
    float *gs = nullptr;  // n_t x k
    float *se = nullptr;  // ring slots x n_t
};

// Row-blocked Q passes of the item pass.  The gathered P table is cut into nb
// blocks of consecutive rows holding about equal shares of the Q pass's cells
// (row_bounds).  In every column bucket x the run of cells whose row falls in
// block j (bounds[j * n_t + x] .. bounds[(j + 1) * n_t + x]) is bucket
// v = j * n_t + x of one combined work plan, in which every block starts on a
// workgroup boundary; one launch runs all blocks, with the workgroups of each
// group of 8 consecutive blocks dealt in turn to the 8 XCDs (the dispatcher's
// order), so that an XCD gathers from its own block of P while the other XCDs
// gather from theirs.  Each bucket's partial sum goes to part[v]; a combine
// kernel adds the nb sums of a column in block order and updates it.  Built
// over the stream the Q pass walks (the other cells' stream when dense tiles
// are on).
struct BlockPlan {
    int32_t nb = 0;
    bool dense = false;
    std::vector<int64_t> hrow_bounds;  // nb + 1 row boundaries (host)
    int64_t *row_bounds = nullptr;     // the same on the device
    int64_t *bounds = nullptr;         // (nb + 1) x n_t
    float *part = nullptr;             // nb x n_t x k
    struct Combined {
        bool ready = false;
        Plan plan;                 // over nb x n_t buckets
        int32_t *sched = nullptr;  // chunk of each workgroup (-1: idle)
        int64_t n_wg = 0;
        float *carry = nullptr;    // one partial sum per wave (carry_per_wave)
    } comb[2];                     // [precision]
};

struct Template {
    int64_t m = 0, n = 0, nnz = 0;
    int32_t m_t = 0, n_t = 0, k = 0;
    int32_t *row_map = nullptr, *col_map = nullptr;
    int2 *stream_r = nullptr, *stream_c = nullptr;
    int64_t *row_ptr = nullptr, *col_ptr = nullptr;
    std::vector<int64_t> hptr[2];  // host copies of row_ptr / col_ptr
    int32_t E = 64;
    Plan plan[2][2];               // [side][precision]
    SlabPlan slab[2];              // [side], fp32 only
    DensePlan dense;               // bf16 only
    bool dense_use = false;        // the current fit runs the dense tiles
    MiniPlan mb;
    SimPlan sim;
    BlockPlan qb;
};

// Epochs whose loss terms are kept before one batched reduction.
constexpr int kLossRing = 16;

struct FitBufs {
    int32_t prec = -1;
    float *P[2] = {nullptr, nullptr}, *Q[2] = {nullptr, nullptr};
    uint16_t *Pb[2] = {nullptr, nullptr}, *Qb[2] = {nullptr, nullptr};
    float *carry_r = nullptr, *carry_c = nullptr, *e2 = nullptr, *normP = nullptr, *normQ = nullptr;
    double *partial = nullptr, *loss = nullptr;
    int32_t loss_cap = 0;
    int64_t item_cap = 0;
};

struct ExtSlot {
    int32_t *fid = nullptr, *free_id = nullptr;
    float *r = nullptr;
    float *X = nullptr;  // the chunk's free rows after the last step
    // Adam extension state (coefficients, moments, partial products, gradients)
    float *Cst = nullptr, *Mst = nullptr, *Vst = nullptr, *qpart = nullptr, *gt = nullptr;
    int64_t adam_cap = 0, qpart_cap = 0, gt_cap = 0;
    hipEvent_t ev_h2d = nullptr, ev_staged = nullptr, ev_done = nullptr, ev_flushed = nullptr;
    // with timing on: start and end of the chunk's copy (copy stream) and of
    // its compute (compute stream); pending until read
    hipEvent_t tm[4] = {nullptr, nullptr, nullptr, nullptr};
    bool tm_pending = false;
};

struct ExtState {
    int64_t cap_nnz = 0;
    int32_t cap_free = 0, k = 0;
    ExtSlot slot[2];
    uint64_t *keys = nullptr, *keys_alt = nullptr;
    uint32_t *vals = nullptr, *vals_alt = nullptr, *sort_scratch = nullptr;
    int2 *stream = nullptr;
    int64_t *ptr = nullptr;
    // work plan of a chunk's item pass (built on the device; the Adam
    // extension's gradient), its bound on the item count and split-bucket sums
    uint32_t *plan_off = nullptr, *plan_nparts = nullptr, *plan_scan = nullptr;
    int32_t *plan_items = nullptr;
    float *plan_carry = nullptr;
    int64_t plan_cap = 0;
    int32_t *err = nullptr;
    uint32_t *unsorted = nullptr;  // the chunk's keys out of order (radix_sort)
    int next = 0;
    bool pending = false;
};

}  // namespace tsid

using namespace tsid;

struct tsid_ctx {
    int device = 0;
    hipStream_t comp = nullptr, h2d = nullptr, d2h = nullptr;
    bool own_comp = false;
    Arena arena;
    std::string err;
    int32_t *err_dev = nullptr;      // error slots of build / fit / loss
    int32_t *err_host = nullptr;     // pinned mirror
    Template *tpl = nullptr;
    int32_t epochs_done = 0;         // of the last fit
    int32_t timing = 0;              // time every timing-th epoch (0: off)
    tsid_timing tm{};
    std::vector<hipEvent_t> events;  // pool of timing events (created by tsid_set_timing, grown on demand)
    size_t events_used = 0;          // pool events handed out in the current fit
    std::vector<hipEvent_t> ev_slot; // this fit's events, kEvents per epoch (null: not timed)
    std::vector<uint8_t> launched;   // which kernel kinds each timed epoch ran
    FitBufs fb;
    ExtState ext;
    int32_t pass_kernel = TSID_PASS_AUTO;
    float dense_fill = -1.f;           // tsid_set_dense_tiles: < 0 auto, 0 off, > 0 fill
    tsid_dense_info dense_used{};       // of the last fit
    int32_t used_kernel[2] = {0, 0};  // pass kernel of each side in the last fit
    int32_t mb_batches = 0;           // tsid_set_minibatch: 0 full-gradient epochs
    uint64_t mb_seed = 0;
    int32_t row_blocks = 0;           // tsid_set_row_blocks: 0 automatic, 1 off, n forced
    int32_t used_blocks = 1;          // row blocks of the last fit's Q pass
    void *noalloc_scratch = nullptr;  // device address of this device's scratch array
};

namespace {

void set_device(const tsid_ctx *c) { TSID_HIP(hipSetDevice(c->device)); }

// Timed kernels of one epoch; each takes a start and an end event attached to
// its dispatch (the loss reduction: start of its first kernel, end of its last).
enum TimedKernel {
    TK_PPASS = 0, TK_PFIX = 1, TK_QPASS = 2, TK_QFIX = 3, TK_REDUCE = 4, TK_PDENSE = 5, TK_QDENSE = 6,
    TK_EPOCH = 7,  // a whole mini-batch epoch (events recorded on the stream around it)
    kTimed = 8
};
constexpr int kEvents = 2 * kTimed;

// Events a fit can draw before the pool grows: created when timing is
// switched on, so that a timed fit creates none while it runs.
constexpr size_t kEventPool = 1024;

void grow_events(tsid_ctx *c, size_t n) {
    while (c->events.size() < n) {
        hipEvent_t e;
        TSID_HIP(hipEventCreate(&e));
        c->events.push_back(e);
    }
}

void ensure_events(tsid_ctx *c, size_t epochs) {
    c->ev_slot.assign(epochs * kEvents, nullptr);
    c->events_used = 0;
    c->launched.assign(epochs, 0);
}

// Events for kernel kind k of epoch ep: a null pair when timing is off or the
// epoch is not sampled.  The loss reduction (one per 16 epochs) is always
// timed while timing is on.
std::pair<hipEvent_t, hipEvent_t> timed(tsid_ctx *c, int ep, int k) {
    if (!c->timing) return {nullptr, nullptr};
    if (k != TK_REDUCE && ep % c->timing != 0) return {nullptr, nullptr};
    c->launched[(size_t)ep] |= (uint8_t)(1u << k);
    const size_t b = (size_t)ep * kEvents + 2 * k;
    if (!c->ev_slot[b]) {  // a pair from the pool (reused if the kernel kind repeats in this epoch)
        grow_events(c, c->events_used + 2);
        c->ev_slot[b] = c->events[c->events_used++];
        c->ev_slot[b + 1] = c->events[c->events_used++];
    }
    return {c->ev_slot[b], c->ev_slot[b + 1]};
}

void collect_timing(tsid_ctx *c, int epochs) {
    auto ev = [&](int ep, int k, int end) { return c->ev_slot[(size_t)ep * kEvents + 2 * k + end]; };
    auto dt = [&](hipEvent_t a, hipEvent_t b) {
        float ms = 0.f;
        TSID_HIP(hipEventElapsedTime(&ms, a, b));
        return (double)ms;
    };
    tsid_timing &t = c->tm;
    for (int ep = 0; ep < epochs; ++ep) {
        const uint8_t l = c->launched[(size_t)ep];
        if (l & (1u << TK_EPOCH)) {
            t.epoch_ms += dt(ev(ep, TK_EPOCH, 0), ev(ep, TK_EPOCH, 1));
            t.epochs += 1;
        }
        for (int k = 0; k < kTimed; ++k) {
            if (!(l & (1u << k)) || k == TK_EPOCH) continue;
            const double ms = dt(ev(ep, k, 0), ev(ep, k, 1));
            if (k == TK_PPASS || k == TK_QPASS) {
                t.pass_ms[k / 2] += ms;
                t.pass_launches[k / 2] += 1;
            } else if (k == TK_REDUCE) {
                t.reduce_ms += ms;
                t.reduce_launches += 1;
            } else if (k == TK_PDENSE || k == TK_QDENSE) {
                t.dense_ms[k == TK_QDENSE] += ms;
                t.dense_launches[k == TK_QDENSE] += 1;
            } else {
                t.fixup_ms += ms;
                t.fixup_launches += 1;
            }
        }
        if (!(l & (1u << TK_PPASS)) || (l & (1u << TK_EPOCH))) continue;  // not a sampled Jacobi epoch
        // an epoch runs dense P, P pass, P fixup, dense Q, Q pass, Q fixup in
        // that order; with both passes in one launch (no Q pass launch of its
        // own): dense P, dense Q, both passes, P fixup, Q fixup
        static const int order1[] = {TK_PDENSE, TK_PPASS, TK_PFIX, TK_QDENSE, TK_QPASS, TK_QFIX};
        static const int order2[] = {TK_PDENSE, TK_QDENSE, TK_PPASS, TK_PFIX, TK_QFIX, TK_QFIX};
        const int *order = (l & (1u << TK_QPASS)) ? order1 : order2;
        int first = -1, end_k = -1;
        for (int j = 0; j < 6; ++j)
            if (l & (1u << order[j])) {
                if (first < 0) first = order[j];
                end_k = order[j];
            }
        t.epoch_ms += dt(ev(ep, first, 0), ev(ep, end_k, 1));
        t.epochs += 1;
    }
}

template <typename F>
tsid_status guarded(tsid_ctx *c, F &&f) {
    if (!c) return TSID_E_INVAL;
    try {
        set_device(c);
        f();
        c->err.clear();
        return TSID_OK;
    } catch (const Error &e) {
        c->err = e.msg;
        return e.st;
    } catch (const std::exception &e) {
        c->err = e.what();
        return TSID_E_DEVICE;
    }
}

void free_dense(tsid_ctx *c, DensePlan &d) {
    Arena &A = c->arena;
    for (int sd = 0; sd < 2; ++sd) {
        A.release(d.tile_ptr[sd]);
        A.release(d.tile_other[sd]);
        A.release(d.R[sd]);
        A.release(d.sparse[sd]);
        A.release(d.sparse_ptr[sd]);
        A.release(d.plan[sd].item_off);
        A.release(d.plan[sd].item_end);
        A.release(d.plan[sd].items);
        A.release(d.gd[sd]);
        A.release(d.seg_tile[sd]);
        A.release(d.seg_order[sd]);
        A.release(d.seg_stripe[sd]);
        A.release(d.stripe_seg[sd]);
        A.release(d.multi[sd]);
        A.release(d.part[sd]);
    }
    d = DensePlan{};
}

void free_plan(tsid_ctx *c, Plan &pl) {
    c->arena.release(pl.item_off);
    c->arena.release(pl.item_end);
    c->arena.release(pl.items);
    pl = Plan{};
}

void free_minibatch(tsid_ctx *c, MiniPlan &mb) {
    for (int sd = 0; sd < 2; ++sd) {
        c->arena.release(mb.stream[sd]);
        c->arena.release(mb.ptr[sd]);
        for (auto &v : mb.plan[sd])
            for (Plan &pl : v) free_plan(c, pl);
    }
    mb = MiniPlan{};
}

void free_sim(tsid_ctx *c, SimPlan &sp) {
    c->arena.release(sp.ptr);
    c->arena.release(sp.col);
    c->arena.release(sp.val);
    c->arena.release(sp.gs);
    c->arena.release(sp.se);
    sp = SimPlan{};
}

void free_blocks(tsid_ctx *c, BlockPlan &qb) {
    c->arena.release(qb.row_bounds);
    c->arena.release(qb.bounds);
    c->arena.release(qb.part);
    for (auto &cb : qb.comb) {
        free_plan(c, cb.plan);
        c->arena.release(cb.sched);
        c->arena.release(cb.carry);
    }
    qb = BlockPlan{};
}

void free_template(tsid_ctx *c, Template *&t) {
    if (!t) return;
    Arena &A = c->arena;
    A.release(t->row_map);
    A.release(t->col_map);
    A.release(t->stream_r);
    A.release(t->stream_c);
    A.release(t->row_ptr);
    A.release(t->col_ptr);
    for (auto &side : t->plan)
        for (Plan &pl : side) {
            A.release(pl.item_off);
            A.release(pl.item_end);
            A.release(pl.items);
        }
    for (SlabPlan &sp : t->slab) {
        A.release(sp.seg);
        A.release(sp.sblk);
        A.release(sp.carry);
    }
    free_dense(c, t->dense);
    free_minibatch(c, t->mb);
    free_sim(c, t->sim);
    free_blocks(c, t->qb);
    delete t;
    t = nullptr;
}

void free_fit(tsid_ctx *c) {
    Arena &A = c->arena;
    FitBufs &f = c->fb;
    for (int b = 0; b < 2; ++b) {
        A.release(f.P[b]);
        A.release(f.Q[b]);
        A.release(f.Pb[b]);
        A.release(f.Qb[b]);
    }
    A.release(f.carry_r);
    A.release(f.carry_c);
    A.release(f.e2);
    A.release(f.normP);
    A.release(f.normQ);
    A.release(f.partial);
    A.release(f.loss);
    f.prec = -1;
    f.loss_cap = 0;
    f.item_cap = 0;
}

void free_ext_buffers(tsid_ctx *c) {
    Arena &A = c->arena;
    ExtState &x = c->ext;
    for (auto &s : x.slot) {
        A.release(s.fid);
        A.release(s.free_id);
        A.release(s.r);
        A.release(s.X);
        A.release(s.Cst);
        A.release(s.Mst);
        A.release(s.Vst);
        A.release(s.qpart);
        A.release(s.gt);
        s.adam_cap = s.qpart_cap = s.gt_cap = 0;
    }
    A.release(x.keys);
    A.release(x.keys_alt);
    A.release(x.vals);
    A.release(x.vals_alt);
    A.release(x.sort_scratch);
    A.release(x.stream);
    A.release(x.ptr);
    A.release(x.plan_off);
    A.release(x.plan_nparts);
    A.release(x.plan_scan);
    A.release(x.plan_items);
    A.release(x.plan_carry);
    x.plan_cap = 0;
    x.cap_nnz = 0;
    x.cap_free = 0;
    x.k = 0;
}

void check_opts(const tsid_fit_opts *o) {
    if (!o) fail(TSID_E_INVAL, "opts is NULL");
    if (o->epochs < 0) fail(TSID_E_INVAL, "epochs < 0");
    if (!(o->lambda >= 0.f) || !std::isfinite(o->lambda)) fail(TSID_E_INVAL, "lambda must be finite and >= 0");
    if (!(o->lr > 0.f) || !std::isfinite(o->lr)) fail(TSID_E_INVAL, "lr must be finite and > 0");
    if (o->clip < 0 || o->clip > 3) fail(TSID_E_INVAL, "clip must be 0, 1, 2 or 3");
    if (o->clip && !(o->clip_xi > 0.f)) fail(TSID_E_INVAL, "clip_xi must be > 0");
    if (o->prec != TSID_FP32 && o->prec != TSID_BF16) fail(TSID_E_INVAL, "bad precision");
    if (o->step != TSID_STEP_SUM && o->step != TSID_STEP_DEGREE && o->step != TSID_STEP_COL_DEGREE)
        fail(TSID_E_INVAL, "bad step");
}

// Whether the rows of `side` (0: rows of R, P; 1: columns, Q) take the
// 1/max(1, deg) step scale of Eq. 5.
int32_t side_scaled(int32_t step, int side) {
    return step == TSID_STEP_DEGREE || (step == TSID_STEP_COL_DEGREE && side == 1);
}

void check_aligned(const void *p, const char *what) {
    if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
        fail(TSID_E_INVAL, std::string(what) + " must be 16-byte aligned");
}

// Validates a template id set on the host: range first, then repeats.
void check_ids(const int32_t *ids, int32_t count, int64_t bound, const char *what) {
    if (count > 0 && !ids) fail(TSID_E_INVAL, std::string(what) + " is NULL");
    for (int32_t a = 0; a < count; ++a)
        if (ids[a] < 0 || ids[a] >= bound) fail(TSID_E_RANGE, std::string(what) + " id out of range");
    std::vector<int32_t> sorted(ids, ids + count);
    std::sort(sorted.begin(), sorted.end());
    if (std::adjacent_find(sorted.begin(), sorted.end()) != sorted.end())
        fail(TSID_E_DUP, std::string(what) + " repeats an id");
}

void raise_device_errors(const int32_t *e, const char *where) {
    if (e[ERR_RANGE]) fail(TSID_E_RANGE, std::string(where) + ": index out of range");
    if (e[ERR_DUP]) fail(TSID_E_DUP, std::string(where) + ": repeated cell");
    if (e[ERR_INVAL]) fail(TSID_E_INVAL, std::string(where) + ": non-finite value");
}

Plan build_plan(tsid_ctx *c, const std::vector<int64_t> &ptr, int32_t rows, int64_t E, int64_t ng);

// E_DUP when a cell (u, i) occurs twice anywhere in Omega: every cell's key
// u * n + i, streamed from the host in pieces of S, sorted on the device, and
// neighbours compared.  Needs 24 bytes per cell of temporary device memory.
void check_omega_unique(tsid_ctx *c, const int32_t *u, const int32_t *i, int64_t nnz, int64_t m, int64_t n,
                        int64_t S) {
    Arena &A = c->arena;
    hipStream_t cs = c->comp;
    uint64_t *keys = nullptr, *alt = nullptr;
    uint32_t *vals = nullptr, *valt = nullptr, *tmp = nullptr;
    int32_t *du = nullptr, *di = nullptr;
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(cs);
        A.release(keys);
        A.release(alt);
        A.release(vals);
        A.release(valt);
        A.release(tmp);
        A.release(du);
        A.release(di);
    };
    try {
        S = std::max<int64_t>(1, std::min<int64_t>(S, nnz));
        keys = A.alloc<uint64_t>(nnz);
        alt = A.alloc<uint64_t>(nnz);
        vals = A.alloc<uint32_t>(nnz);
        valt = A.alloc<uint32_t>(nnz);
        tmp = A.alloc<uint32_t>((int64_t)radix_scratch_elems(nnz));
        du = A.alloc<int32_t>(S);
        di = A.alloc<int32_t>(S);
        for (int64_t p0 = 0; p0 < nnz; p0 += S) {
            const int64_t len = std::min<int64_t>(S, nnz - p0);
            TSID_HIP(hipMemcpyAsync(du, u + p0, (size_t)len * 4, hipMemcpyHostToDevice, cs));
            TSID_HIP(hipMemcpyAsync(di, i + p0, (size_t)len * 4, hipMemcpyHostToDevice, cs));
            cell_keys(du, di, len, n, keys + p0, vals + p0, cs);
        }
        const bool in_alt = radix_sort(keys, vals, alt, valt, nnz, bits_for(m * n), tmp, cs);
        TSID_HIP(hipMemsetAsync(c->err_dev, 0, ERR_SLOTS * sizeof(int32_t), cs));
        adjacent_equal(in_alt ? alt : keys, nnz, c->err_dev, cs);
        TSID_HIP(hipMemcpyAsync(c->err_host, c->err_dev, ERR_SLOTS * 4, hipMemcpyDeviceToHost, cs));
        TSID_HIP(hipStreamSynchronize(cs));
        if (c->err_host[ERR_DUP]) fail(TSID_E_DUP, "build: a cell (u, i) occurs twice in Omega");
    } catch (...) {
        cleanup();
        throw;
    }
    cleanup();
}

void build(tsid_ctx *c, int64_t m, int64_t n, const int32_t *u, const int32_t *i, const float *r,
           int64_t nnz, const int32_t *I, int32_t m_t, const int32_t *J, int32_t n_t, int32_t k,
           int64_t stage) {
    if (m < 1 || n < 1 || m >= (int64_t(1) << 31) || n >= (int64_t(1) << 31))
        fail(TSID_E_INVAL, "m and n must be in [1, 2^31)");
    if (nnz < 0) fail(TSID_E_INVAL, "nnz < 0");
    if (nnz > 0 && (!u || !i || !r)) fail(TSID_E_INVAL, "NULL Omega arrays");
    if (m_t < 0 || m_t > m || n_t < 0 || n_t > n) fail(TSID_E_INVAL, "template size out of range");
    if (!valid_rank(k)) fail(TSID_E_INVAL, "k must be 8, 16, 32, 64 or 128");
    if (stage < 0) fail(TSID_E_INVAL, "stage_entries < 0");
    check_ids(I, m_t, m, "I");
    check_ids(J, n_t, n, "J");

    hipStream_t cs = c->comp, hs = c->h2d;
    Arena &A = c->arena;
    Template *t = new Template;
    t->m = m;
    t->n = n;
    t->m_t = m_t;
    t->n_t = n_t;
    t->k = k;
    // Scratch memory of the template construction; released on every path.
    int32_t *dI = nullptr, *dJ = nullptr, *su[2] = {nullptr, nullptr}, *si[2] = {nullptr, nullptr};
    float *sr[2] = {nullptr, nullptr};
    uint32_t *bcnt = nullptr, *boffs = nullptr, *piece = nullptr, *scan_tmp = nullptr;
    uint32_t *sort_tmp = nullptr, *vals = nullptr, *vals_alt = nullptr;
    uint64_t *keys = nullptr, *keys_alt = nullptr;
    uint32_t *piece_host = nullptr;
    hipEvent_t ev_h2d[2] = {nullptr, nullptr}, ev_free[2] = {nullptr, nullptr};
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(hs);
        (void)hipStreamSynchronize(cs);
        A.release(dI);
        A.release(dJ);
        for (int s = 0; s < 2; ++s) {
            A.release(su[s]);
            A.release(si[s]);
            A.release(sr[s]);
            if (ev_h2d[s]) (void)hipEventDestroy(ev_h2d[s]);
            if (ev_free[s]) (void)hipEventDestroy(ev_free[s]);
        }
        A.release(bcnt);
        A.release(boffs);
        A.release(piece);
        A.release(scan_tmp);
        A.release(sort_tmp);
        A.release(keys);
        A.release(keys_alt);
        A.release(vals);
        A.release(vals_alt);
        if (piece_host) (void)hipHostFree(piece_host);
    };
    try {
        // a1: template maps
        t->row_map = A.alloc<int32_t>(m);
        t->col_map = A.alloc<int32_t>(n);
        fill_i32(t->row_map, m, -1, cs);
        fill_i32(t->col_map, n, -1, cs);
        dI = A.alloc<int32_t>(m_t);
        dJ = A.alloc<int32_t>(n_t);
        if (m_t) TSID_HIP(hipMemcpyAsync(dI, I, (size_t)m_t * 4, hipMemcpyHostToDevice, cs));
        if (n_t) TSID_HIP(hipMemcpyAsync(dJ, J, (size_t)n_t * 4, hipMemcpyHostToDevice, cs));
        scatter_map(dI, m_t, t->row_map, cs);
        scatter_map(dJ, n_t, t->col_map, cs);
        TSID_HIP(hipMemsetAsync(c->err_dev, 0, ERR_SLOTS * sizeof(int32_t), cs));

        // a2: stream Omega through two staging slots; filter each piece to Omega*.
        const int bits_a = bits_for(m_t), bits_b = bits_for(n_t);
        const int64_t S = std::max<int64_t>(1, std::min<int64_t>(stage ? stage : kDefaultStage,
                                                                 std::max<int64_t>(nnz, 1)));
        const int64_t pieces = nnz > 0 ? (nnz + S - 1) / S : 0;
        const int nfb = filter_blocks(S);
        bcnt = A.alloc<uint32_t>(nfb);
        boffs = A.alloc<uint32_t>(nfb);
        piece = A.alloc<uint32_t>(1);
        scan_tmp = A.alloc<uint32_t>((int64_t)scan_scratch_elems(std::max<int64_t>(nfb, m_t + n_t + 1)));
        TSID_HIP(hipHostMalloc((void **)&piece_host, sizeof(uint32_t), hipHostMallocDefault));
        int64_t cap = pieces ? std::min<int64_t>(nnz, std::max<int64_t>(S, int64_t(1) << 20)) : 1;
        keys = A.alloc<uint64_t>(cap);
        vals = A.alloc<uint32_t>(cap);
        int64_t total = 0;
        if (pieces) {
            for (int s = 0; s < 2 && s < pieces; ++s) {
                su[s] = A.alloc<int32_t>(S);
                si[s] = A.alloc<int32_t>(S);
                sr[s] = A.alloc<float>(S);
                TSID_HIP(hipEventCreateWithFlags(&ev_h2d[s], hipEventDisableTiming));
                TSID_HIP(hipEventCreateWithFlags(&ev_free[s], hipEventDisableTiming));
            }
            auto issue = [&](int64_t p) {
                const int s = (int)(p & 1);
                const int64_t off = p * S, len = std::min(S, nnz - off);
                TSID_HIP(hipStreamWaitEvent(hs, ev_free[s], 0));
                TSID_HIP(hipMemcpyAsync(su[s], u + off, (size_t)len * 4, hipMemcpyHostToDevice, hs));
                TSID_HIP(hipMemcpyAsync(si[s], i + off, (size_t)len * 4, hipMemcpyHostToDevice, hs));
                TSID_HIP(hipMemcpyAsync(sr[s], r + off, (size_t)len * 4, hipMemcpyHostToDevice, hs));
                TSID_HIP(hipEventRecord(ev_h2d[s], hs));
            };
            issue(0);
            for (int64_t p = 0; p < pieces; ++p) {
                const int s = (int)(p & 1);
                const int64_t len = std::min(S, nnz - p * S);
                if (p + 1 < pieces) issue(p + 1);  // overlaps this piece's filter
                TSID_HIP(hipStreamWaitEvent(cs, ev_h2d[s], 0));
                filter_count(su[s], si[s], sr[s], len, t->row_map, t->col_map, m, n, bcnt,
                             c->err_dev, cs);
                const int nb = filter_blocks(len);
                scan_u32(bcnt, boffs, nb, piece, scan_tmp, cs);
                TSID_HIP(hipMemcpyAsync(piece_host, piece, 4, hipMemcpyDeviceToHost, cs));
                TSID_HIP(hipStreamSynchronize(cs));
                const int64_t got = *piece_host;
                if (total + got > kMaxEntries) fail(TSID_E_INVAL, "template holds more than 2^32-1 cells");
                if (total + got > cap) {  // grow the output, keeping what is there
                    int64_t ncap = std::max<int64_t>(total + got, std::min<int64_t>(nnz, cap * 2));
                    uint64_t *nk = A.alloc<uint64_t>(ncap);
                    uint32_t *nv = A.alloc<uint32_t>(ncap);
                    if (total) {
                        TSID_HIP(hipMemcpyAsync(nk, keys, (size_t)total * 8, hipMemcpyDeviceToDevice, cs));
                        TSID_HIP(hipMemcpyAsync(nv, vals, (size_t)total * 4, hipMemcpyDeviceToDevice, cs));
                        TSID_HIP(hipStreamSynchronize(cs));
                    }
                    A.release(keys);
                    A.release(vals);
                    keys = nk;
                    vals = nv;
                    cap = ncap;
                }
                filter_write(su[s], si[s], sr[s], len, t->row_map, t->col_map, m, n, boffs, total,
                             bits_b, keys, vals, cs);
                TSID_HIP(hipEventRecord(ev_free[s], cs));
                total += got;
            }
        }
        t->nnz = total;

        // a3: buckets by row (CSR, key a<<bits_b|b) and by column (CSC, key b<<bits_a|a).
        keys_alt = A.alloc<uint64_t>(total);
        vals_alt = A.alloc<uint32_t>(total);
        sort_tmp = A.alloc<uint32_t>((int64_t)radix_scratch_elems(total));
        const int nbits = bits_a + bits_b;
        bool in_alt = radix_sort(keys, vals, keys_alt, vals_alt, total, nbits, sort_tmp, cs);
        uint64_t *ck = in_alt ? keys_alt : keys;
        uint32_t *cv = in_alt ? vals_alt : vals;
        t->stream_r = A.alloc<int2>(total);
        t->row_ptr = A.alloc<int64_t>((int64_t)m_t + 1);
        keys_to_stream(ck, cv, total, bits_b, t->stream_r, c->err_dev, cs);
        ptr_from_keys(ck, total, m_t, bits_b, t->row_ptr, cs);
        uint64_t *ok = in_alt ? keys : keys_alt;
        uint32_t *ov = in_alt ? vals : vals_alt;
        swap_key_halves(ck, total, bits_b, bits_a, ok, cs);
        if (total) TSID_HIP(hipMemcpyAsync(ov, cv, (size_t)total * 4, hipMemcpyDeviceToDevice, cs));
        // sort (ok, ov) using (ck, cv) as the other buffer
        bool alt2 = radix_sort(ok, ov, ck, cv, total, nbits, sort_tmp, cs);
        uint64_t *tk = alt2 ? ck : ok;
        uint32_t *tv = alt2 ? cv : ov;
        t->stream_c = A.alloc<int2>(total);
        t->col_ptr = A.alloc<int64_t>((int64_t)n_t + 1);
        keys_to_stream(tk, tv, total, bits_a, t->stream_c, c->err_dev, cs);
        ptr_from_keys(tk, total, n_t, bits_a, t->col_ptr, cs);

        // host copies of the bucket pointers, for the work plans built at fit time
        t->E = choose_E(total);
        t->hptr[0].resize((size_t)m_t + 1);
        t->hptr[1].resize((size_t)n_t + 1);
        TSID_HIP(hipMemcpyAsync(t->hptr[0].data(), t->row_ptr, ((size_t)m_t + 1) * 8,
                                hipMemcpyDeviceToHost, cs));
        TSID_HIP(hipMemcpyAsync(t->hptr[1].data(), t->col_ptr, ((size_t)n_t + 1) * 8,
                                hipMemcpyDeviceToHost, cs));
        TSID_HIP(hipMemcpyAsync(c->err_host, c->err_dev, ERR_SLOTS * 4, hipMemcpyDeviceToHost, cs));
        TSID_HIP(hipStreamSynchronize(cs));
        raise_device_errors(c->err_host, "build");
        // the fp32 work plan of the row side comes with the template: the
        // loss needs it, and tsid_loss_noalloc may not allocate it later
        t->plan[0][TSID_FP32] = build_plan(c, t->hptr[0], m_t, t->E, items_per_wave(k, TSID_FP32));
    } catch (...) {
        cleanup();
        free_template(c, t);
        throw;
    }
    cleanup();
    // Omega is a set (Definition 1).  The template's own check sees repeats
    // among its cells only; when cells fall outside it, all of Omega is
    // checked as well.
    if (t->nnz < nnz) {
        try {
            check_omega_unique(c, u, i, nnz, m, n, stage ? stage : kDefaultStage);
        } catch (...) {
            free_template(c, t);
            throw;
        }
    }
    free_template(c, c->tpl);
    free_fit(c);
    c->tpl = t;
}

// Work plan of one pass: bucket x becomes p items of at most E cells, where p
// is max(1, ceil(deg / E)) rounded up to a power of two while it fits a wave
// (ng groups), else to a multiple of ng.  Buckets of p <= ng items start at a
// multiple of p (idle pad items fill the gaps), so they never straddle two
// waves and their partial sums are combined inside the pass; only buckets of
// more than one wave leave partial sums for the fixup kernel.
// The host layout of such a plan: off / endv (rows + 1) and items; returns
// the item length it settled on.
struct PlanLayout {
    std::vector<uint32_t> off, endv;
    std::vector<int32_t> items;
    int64_t E = 64;
    bool spans = false;
};
PlanLayout layout_plan(const std::vector<int64_t> &ptr, int32_t rows, int64_t E, int64_t ng) {
    int64_t maxdeg = 0;
    for (int32_t x = 0; x < rows; ++x) maxdeg = std::max(maxdeg, ptr[x + 1] - ptr[x]);
    // When items up to twice the default length keep every bucket within one
    // wave, take them: no bucket then needs the fixup kernel.
    if (maxdeg > E * ng) {
        const int64_t e1 = ((maxdeg + ng - 1) / ng + 15) / 16 * 16;
        if (e1 <= 2 * E) E = e1;
    }
    PlanLayout L;
    L.off.resize((size_t)rows + 1);
    L.endv.resize((size_t)rows + 1);
    int64_t cur = 0;
    for (int32_t x = 0; x < rows; ++x) {
        const int64_t deg = ptr[x + 1] - ptr[x];
        int64_t p = deg <= E ? 1 : (deg + E - 1) / E;
        if (p > 1 && p <= ng) {
            int64_t q = 1;
            while (q < p) q <<= 1;
            p = q;
        } else if (p > ng) {
            p = (p + ng - 1) / ng * ng;
            L.spans = true;
        }
        const int64_t align = p < ng ? p : ng;
        const int64_t start = (cur + align - 1) / align * align;
        L.items.resize((size_t)(start + p), -1);
        for (int64_t j = start; j < start + p; ++j) L.items[(size_t)j] = x;
        L.off[(size_t)x] = (uint32_t)start;
        L.endv[(size_t)x] = (uint32_t)(start + p);
        cur = start + p;
    }
    if (cur >= INT32_MAX) fail(TSID_E_INVAL, "work plan too large");
    L.E = E;
    return L;
}

Plan upload_plan(tsid_ctx *c, const PlanLayout &L, int32_t rows) {
    const int64_t cur = (int64_t)L.items.size();
    Arena &A = c->arena;
    uint32_t *d_off = nullptr, *d_end = nullptr;
    int32_t *d_items = nullptr;
    try {
        d_off = A.alloc<uint32_t>((int64_t)rows + 1);
        d_end = A.alloc<uint32_t>((int64_t)rows + 1);
        d_items = A.alloc<int32_t>(cur);
        hipStream_t cs = c->comp;
        TSID_HIP(hipMemcpyAsync(d_off, L.off.data(), ((size_t)rows + 1) * 4, hipMemcpyHostToDevice, cs));
        TSID_HIP(hipMemcpyAsync(d_end, L.endv.data(), ((size_t)rows + 1) * 4, hipMemcpyHostToDevice, cs));
        if (cur) TSID_HIP(hipMemcpyAsync(d_items, L.items.data(), (size_t)cur * 4, hipMemcpyHostToDevice, cs));
        TSID_HIP(hipStreamSynchronize(cs));  // the host vectors may go out of scope
    } catch (...) {
        A.release(d_off);
        A.release(d_end);
        A.release(d_items);
        throw;
    }
    Plan pl;
    pl.item_off = d_off;
    pl.item_end = d_end;
    pl.items = d_items;
    pl.n_items = (int32_t)cur;
    pl.E = (int32_t)L.E;
    pl.spans = L.spans;
    pl.ready = true;
    return pl;
}

Plan build_plan(tsid_ctx *c, const std::vector<int64_t> &ptr, int32_t rows, int64_t E, int64_t ng) {
    return upload_plan(c, layout_plan(ptr, rows, E, ng), rows);
}

void ensure_plan(tsid_ctx *c, int side, int prec) {
    Template &t = *c->tpl;
    Plan &pl = t.plan[side][prec];
    if (pl.ready) return;
    const int32_t rows = side ? t.n_t : t.m_t;
    pl = build_plan(c, t.hptr[side], rows, t.E, items_per_wave(t.k, prec));
}

// Whether the slab pass suits one side of the template: the expected number
// of cells per slab row and block of owner rows (the LDS reuse of a staged
// row) is at least 4, and no bucket is much longer than the mean, since one
// lane walks a whole bucket.  (The item pass takes the rest.)
#ifndef TSID_SLAB_MIN_REUSE
#define TSID_SLAB_MIN_REUSE 4.0
#endif
bool slab_suits(const Template &t, int side) {
    const int64_t rows = side ? t.n_t : t.m_t, y_rows = side ? t.m_t : t.n_t;
    if (rows < 1 || y_rows < 1 || t.nnz < 1) return false;
    const double density = (double)t.nnz / ((double)rows * (double)y_rows);
    if (density * kSlabLanes < TSID_SLAB_MIN_REUSE) return false;
    const std::vector<int64_t> &ptr = t.hptr[side];
    int64_t maxdeg = 0;
    for (int64_t x = 0; x < rows; ++x) maxdeg = std::max(maxdeg, ptr[(size_t)x + 1] - ptr[(size_t)x]);
    const double mean = (double)t.nnz / (double)rows;
    return (double)maxdeg <= 2.0 * mean + 64.0;
}

// Workgroups one side's slab pass aims for: the `sides` passes of an epoch
// (one launch) together fill one round of the compute units, with as many
// resident workgroups per unit as its LDS holds slabs.  TSID_SLAB_UNITS, a
// tuning knob, sets the count per side instead.
int64_t slab_target_units(int device, int sides) {
    if (const char *e = std::getenv("TSID_SLAB_UNITS")) {
        const long v = std::strtol(e, nullptr, 10);
        if (v > 0) return v;
    }
    int cus = 0, lds = 0;
    TSID_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device));
    TSID_HIP(hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device));
    return std::max<int64_t>(1, (int64_t)std::max(1, cus) * std::max(1, lds / kSlabBytes) / std::max(1, sides));
}

// Whether side `side` runs the slab pass in this fit (from the pass-kernel
// mode and the precision).
bool slab_wanted(tsid_ctx *c, int side, int prec) {
    Template &t = *c->tpl;
    SlabPlan &sp = t.slab[side];
    const int mode = c->pass_kernel;
    bool want = false;
    if (mode == TSID_PASS_SLAB) {
        if (!slab_supported(t.k, prec))
            fail(TSID_E_INVAL, "the slab pass needs fp32 factors and k in {8, 16, 32, 64}");
        want = true;
    } else if (mode == TSID_PASS_AUTO) {
        if (sp.suits < 0) sp.suits = slab_supported(t.k, TSID_FP32) && slab_suits(t, side);
        want = sp.suits == 1 && prec == TSID_FP32;
    }
    const int32_t rows = side ? t.n_t : t.m_t, y_rows = side ? t.m_t : t.n_t;
    return want && rows > 0 && y_rows > 0;  // an empty side has no cells: the item pass shrinks it
}

// Sets whether side `side` runs the slab pass (`want`), and builds its plan
// the first time it does.  `sides`: how many sides run it; their passes
// share one launch, so together they aim for one round of the compute units.
void ensure_slab(tsid_ctx *c, int side, bool want, int sides) {
    Template &t = *c->tpl;
    SlabPlan &sp = t.slab[side];
    const int32_t rows = side ? t.n_t : t.m_t, y_rows = side ? t.m_t : t.n_t;
    if (want && !sp.ready) {
        Arena &A = c->arena;
        hipStream_t cs = c->comp;
        const int32_t C = slab_rows(t.k);
        const int32_t n_slabs = std::max(1, ceil_div(y_rows, C));
        const int32_t n_blocks = ceil_div(rows, kSlabLanes);
        const int64_t u_target = std::max<int64_t>(1, slab_target_units(c->device, sides) / n_blocks);
        const int32_t S = ceil_div(n_slabs, std::min<int64_t>(u_target, n_slabs));
        const int32_t U = ceil_div(n_slabs, S);
        uint32_t *seg = nullptr, *pseg = nullptr;
        uint4 *sblk = nullptr;
        float *carry = nullptr;
        try {
            // the runs (x, s) of the bucketed stream, then their places in the
            // pass's copy: slab-major, each padded to a multiple of 8 records
            const int64_t nr = (int64_t)n_slabs * rows;
            seg = A.alloc<uint32_t>(nr + rows);
            const int2 *src = side ? t.stream_c : t.stream_r;
            launch_slab_seg(src, side ? t.col_ptr : t.row_ptr, rows, n_slabs, C, seg, cs);
            std::vector<uint32_t> hs((size_t)(nr + rows)), hp((size_t)nr + 1);
            TSID_HIP(hipMemcpyAsync(hs.data(), seg, hs.size() * 4, hipMemcpyDeviceToHost, cs));
            TSID_HIP(hipStreamSynchronize(cs));
            int64_t pos = 0;
            for (int64_t r = 0; r < nr; ++r) {
                hp[(size_t)r] = (uint32_t)pos;
                pos += ((int64_t)(hs[(size_t)(r + rows)] - hs[(size_t)r]) + 7) / 8 * 8;
                if (pos > (int64_t)UINT32_MAX) fail(TSID_E_INVAL, "slab stream too long for 32-bit pointers");
            }
            hp[(size_t)nr] = (uint32_t)pos;
            pseg = A.alloc<uint32_t>(nr + 1);
            sblk = A.alloc<uint4>(std::max<int64_t>(pos / 8 * 3, 3));  // 48 bytes per 8 records
            if (U > 1) carry = A.alloc<float>((int64_t)n_blocks * U * kSlabLanes * t.k);
            TSID_HIP(hipMemcpyAsync(pseg, hp.data(), hp.size() * 4, hipMemcpyHostToDevice, cs));
            launch_slab_order(src, seg, rows, n_slabs, C, pseg, sblk, cs);
            TSID_HIP(hipStreamSynchronize(cs));
            A.release(seg);
            seg = nullptr;
        } catch (...) {
            A.release(seg);
            A.release(pseg);
            A.release(sblk);
            A.release(carry);
            throw;
        }
        sp.seg = pseg;
        sp.sblk = sblk;
        sp.carry = carry;
        sp.C = C;
        sp.n_slabs = n_slabs;
        sp.n_blocks = n_blocks;
        sp.S = S;
        sp.U = U;
        sp.ready = true;
    }
    sp.use = want;
}

// Work segments of one side: a stripe's tile list is cut into
// ceil(len / L) near-equal runs of consecutive tiles, L = max(seg_min,
// ceil(len / seg_max)), so that a long stripe (a Zipf head row block meets
// nearly every other block) spreads over up to seg_max waves and a short one
// takes one.  Also counts the stripes that hold a tile.
#ifndef TSID_DENSE_SEG_MIN
#define TSID_DENSE_SEG_MIN 32
#endif
#ifndef TSID_DENSE_SEG_MAX
#define TSID_DENSE_SEG_MAX 64
#endif
// The segments of one side's stripes and their launch order.  The other
// side's tiles are cut into `ranges` equal ranges, and the segments are
// launched by the range their first tile lies in, then in stripe order, so
// the waves running together gather the other factor's rows from one range
// of its table; ranges = 0 keeps plain stripe order, in which the segments of
// a stripe read their tile values in sequence, and ranges at least the
// number of other-side tiles sorts by the first tile itself.  Measured on
// Billion-scale: the P side (gathering from the 25.6 MB Q table) 1.31 ms in
// stripe order, 1.29-1.31 with 8 to 64 ranges, 1.24 sorted by the first
// tile; the Q side (gathering from 256 MB of P) 1.54 ms in stripe order and
// 1.71-1.88 with any ranges.  Tuning knobs TSID_DENSE_RANGES_P / _Q.
#ifndef TSID_DENSE_RANGES_P
#define TSID_DENSE_RANGES_P 65536
#endif
#ifndef TSID_DENSE_RANGES_Q
#define TSID_DENSE_RANGES_Q 0
#endif
void dense_segments(tsid_ctx *c, DensePlan &d, int sd, const std::vector<uint32_t> &tp,
                    const std::vector<int32_t> &tile_other) {
    const int64_t n_st = (int64_t)tp.size() - 1;
    std::vector<uint32_t> seg_tile, stripe_seg((size_t)n_st + 1);
    std::vector<int32_t> seg_stripe, multi;
    for (int64_t x = 0; x < n_st; ++x) {
        stripe_seg[(size_t)x] = (uint32_t)seg_stripe.size();
        const int64_t len = (int64_t)tp[(size_t)x + 1] - tp[(size_t)x];
        if (len <= 0) continue;
        d.stripes[sd] += 1;
        const int64_t L = std::max<int64_t>(TSID_DENSE_SEG_MIN, (len + TSID_DENSE_SEG_MAX - 1) / TSID_DENSE_SEG_MAX);
        const int64_t n = (len + L - 1) / L;
        for (int64_t q = 0; q < n; ++q) {
            seg_tile.push_back(tp[(size_t)x] + (uint32_t)(q * len / n));
            seg_stripe.push_back((int32_t)x);
        }
        if (n > 1) multi.push_back((int32_t)x);
    }
    stripe_seg[(size_t)n_st] = (uint32_t)seg_stripe.size();
    seg_tile.push_back(tp[(size_t)n_st]);
    Arena &A = c->arena;
    hipStream_t cs = c->comp;
    const int64_t ns = (int64_t)seg_stripe.size();
    std::vector<int32_t> order((size_t)ns);
    for (int64_t q = 0; q < ns; ++q) order[(size_t)q] = (int32_t)q;
    const char *re = std::getenv(sd ? "TSID_DENSE_RANGES_Q" : "TSID_DENSE_RANGES_P");
    const int64_t ranges = re ? std::atoll(re) : (sd ? TSID_DENSE_RANGES_Q : TSID_DENSE_RANGES_P);
    if (ranges > 0 && ns > 0) {
        const int64_t n_other = (sd ? c->tpl->m_t + 15 : c->tpl->n_t + 15) / 16;  // other-side tiles
        auto range_of = [&](int32_t g) {
            return (int64_t)tile_other[seg_tile[(size_t)g]] * ranges / std::max<int64_t>(1, n_other);
        };
        std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return range_of(a) < range_of(b); });
    }
    d.seg_order[sd] = A.alloc<int32_t>(std::max<int64_t>(ns, 1));
    if (ns) TSID_HIP(hipMemcpyAsync(d.seg_order[sd], order.data(), (size_t)ns * 4, hipMemcpyHostToDevice, cs));
    d.n_segs[sd] = ns;
    d.n_multi[sd] = (int64_t)multi.size();
    d.seg_tile[sd] = A.alloc<uint32_t>(ns + 1);
    d.seg_stripe[sd] = A.alloc<int32_t>(std::max<int64_t>(ns, 1));
    d.stripe_seg[sd] = A.alloc<uint32_t>(n_st + 1);
    d.multi[sd] = A.alloc<int32_t>(std::max<int64_t>(d.n_multi[sd], 1));
    d.part[sd] = d.n_multi[sd] ? A.alloc<float>(ns * 16 * c->tpl->k) : nullptr;
    TSID_HIP(hipMemcpyAsync(d.seg_tile[sd], seg_tile.data(), seg_tile.size() * 4, hipMemcpyHostToDevice, cs));
    if (ns)
        TSID_HIP(hipMemcpyAsync(d.seg_stripe[sd], seg_stripe.data(), (size_t)ns * 4, hipMemcpyHostToDevice, cs));
    TSID_HIP(hipMemcpyAsync(d.stripe_seg[sd], stripe_seg.data(), stripe_seg.size() * 4, hipMemcpyHostToDevice, cs));
    if (!multi.empty())
        TSID_HIP(hipMemcpyAsync(d.multi[sd], multi.data(), multi.size() * 4, hipMemcpyHostToDevice, cs));
    TSID_HIP(hipStreamSynchronize(cs));  // the host vectors go out of scope
}

// Builds the dense head tiles of the template for tile fill `fill` (a tile is
// dense when it holds at least ceil(fill * 256) cells): tile counts, flags and
// their prefix sums in both orientations, the tile lists, the owner-major
// tile values, the sparse streams of the other cells with their pointers and
// work plans, and the dense gradient buffers.
void build_dense(tsid_ctx *c, float fill) {
    Template &t = *c->tpl;
    DensePlan &d = t.dense;
    free_dense(c, d);
    Arena &A = c->arena;
    hipStream_t cs = c->comp;
    const int K = t.k;
    const int64_t n_ti = (t.m_t + 15) / 16, n_tj = (t.n_t + 15) / 16, NT = n_ti * n_tj;
    const uint32_t thr = std::max<uint32_t>(1u, (uint32_t)std::ceil(fill * 256.f));
    uint32_t *cnt = nullptr, *flag_p = nullptr, *idx_p = nullptr, *flag_q = nullptr, *idx_q = nullptr;
    uint32_t *scratch = nullptr, *total = nullptr;
    int64_t *cnt_sp[2] = {nullptr, nullptr};
    auto cleanup = [&]() {
        (void)hipStreamSynchronize(cs);
        A.release(cnt);
        A.release(flag_p);
        A.release(idx_p);
        A.release(flag_q);
        A.release(idx_q);
        A.release(scratch);
        A.release(total);
        A.release(cnt_sp[0]);
        A.release(cnt_sp[1]);
    };
    try {
        d.fill = fill;
        if (NT > 0 && t.nnz > 0) {
            cnt = A.alloc<uint32_t>(NT);
            flag_p = A.alloc<uint32_t>(NT);
            idx_p = A.alloc<uint32_t>(NT);
            flag_q = A.alloc<uint32_t>(NT);
            idx_q = A.alloc<uint32_t>(NT);
            scratch = A.alloc<uint32_t>((int64_t)scan_scratch_elems(NT));
            total = A.alloc<uint32_t>(2);
            TSID_HIP(hipMemsetAsync(cnt, 0, (size_t)NT * 4, cs));
            tile_count(t.stream_r, t.row_ptr, t.m_t, n_tj, cnt, cs);
            tile_flag(cnt, n_ti, n_tj, thr, false, flag_p, cs);
            scan_u32(flag_p, idx_p, NT, total, scratch, cs);
            tile_flag(cnt, n_ti, n_tj, thr, true, flag_q, cs);
            scan_u32(flag_q, idx_q, NT, total + 1, scratch, cs);
            uint32_t h_total = 0;
            TSID_HIP(hipMemcpyAsync(&h_total, total, 4, hipMemcpyDeviceToHost, cs));
            TSID_HIP(hipStreamSynchronize(cs));
            d.tiles = h_total;
        }
        const int64_t nd = d.tiles;
        const int32_t rows[2] = {t.m_t, t.n_t};
        const int64_t stripes[2] = {n_ti, n_tj}, others[2] = {n_tj, n_ti};
        for (int sd = 0; sd < 2; ++sd) {
            d.tile_ptr[sd] = A.alloc<uint32_t>(stripes[sd] + 1);
            d.tile_other[sd] = A.alloc<int32_t>(std::max<int64_t>(nd, 1));
            d.R[sd] = A.alloc<float>(std::max<int64_t>(nd, 1) * 256);
            d.gd[sd] = A.alloc<float>((int64_t)rows[sd] * K);
            d.sparse_ptr[sd] = A.alloc<int64_t>((int64_t)rows[sd] + 1);
            cnt_sp[sd] = A.alloc<int64_t>(std::max<int32_t>(rows[sd], 1));
        }
        std::vector<int64_t> hsp[2];
        if (nd > 0) {
            tile_list(flag_p, idx_p, n_ti, n_tj, d.tile_other[0], d.tile_ptr[0], cs);
            tile_list(flag_q, idx_q, n_tj, n_ti, d.tile_other[1], d.tile_ptr[1], cs);
            for (int sd = 0; sd < 2; ++sd) {
                std::vector<uint32_t> tp((size_t)stripes[sd] + 1);
                TSID_HIP(hipMemcpyAsync(tp.data(), d.tile_ptr[sd], (size_t)stripes[sd] * 4, hipMemcpyDeviceToHost,
                                        cs));
                TSID_HIP(hipStreamSynchronize(cs));
                tp[(size_t)stripes[sd]] = (uint32_t)nd;
                std::vector<int32_t> to((size_t)nd);
                TSID_HIP(hipMemcpyAsync(to.data(), d.tile_other[sd], (size_t)nd * 4, hipMemcpyDeviceToHost, cs));
                TSID_HIP(hipStreamSynchronize(cs));
                dense_segments(c, d, sd, tp, to);
            }
            fill_nan(d.R[0], nd * 256, cs);
            fill_nan(d.R[1], nd * 256, cs);
            sparse_count(t.stream_r, t.row_ptr, t.m_t, 0, n_tj, flag_p, cnt_sp[0], cs);
            sparse_count(t.stream_c, t.col_ptr, t.n_t, 1, n_tj, flag_p, cnt_sp[1], cs);
        }
        const uint32_t h_nd = (uint32_t)nd;
        for (int sd = 0; sd < 2; ++sd) {
            TSID_HIP(hipMemcpyAsync(d.tile_ptr[sd] + stripes[sd], &h_nd, 4, hipMemcpyHostToDevice, cs));
            if (nd == 0) TSID_HIP(hipMemsetAsync(d.tile_ptr[sd], 0, (size_t)stripes[sd] * 4, cs));
            std::vector<int64_t> cnt_h((size_t)rows[sd]);
            if (nd > 0 && rows[sd] > 0) {
                TSID_HIP(hipMemcpyAsync(cnt_h.data(), cnt_sp[sd], (size_t)rows[sd] * 8, hipMemcpyDeviceToHost, cs));
            } else {
                for (int32_t x = 0; x < rows[sd]; ++x) cnt_h[(size_t)x] = t.hptr[sd][x + 1] - t.hptr[sd][x];
            }
            TSID_HIP(hipStreamSynchronize(cs));
            hsp[sd].resize((size_t)rows[sd] + 1);
            hsp[sd][0] = 0;
            for (int32_t x = 0; x < rows[sd]; ++x) hsp[sd][x + 1] = hsp[sd][x] + cnt_h[(size_t)x];
            TSID_HIP(hipMemcpyAsync(d.sparse_ptr[sd], hsp[sd].data(), ((size_t)rows[sd] + 1) * 8,
                                    hipMemcpyHostToDevice, cs));
            d.sparse[sd] = A.alloc<int2>(std::max<int64_t>(hsp[sd][(size_t)rows[sd]], 1));
        }
        d.sparse_nnz = hsp[0][(size_t)t.m_t];
        d.cells = t.nnz - d.sparse_nnz;
        if (nd > 0) {
            tile_split(t.stream_r, t.row_ptr, t.m_t, 0, n_ti, n_tj, flag_p, idx_p, flag_q, idx_q, d.R[0], d.R[1],
                       d.sparse_ptr[0], d.sparse[0], cs);
            tile_split(t.stream_c, t.col_ptr, t.n_t, 1, n_ti, n_tj, flag_p, idx_p, flag_q, idx_q, d.R[0], d.R[1],
                       d.sparse_ptr[1], d.sparse[1], cs);
        } else {
            for (int sd = 0; sd < 2; ++sd)
                if (t.nnz)
                    TSID_HIP(hipMemcpyAsync(d.sparse[sd], sd ? t.stream_c : t.stream_r, (size_t)t.nnz * 8,
                                            hipMemcpyDeviceToDevice, cs));
        }
        TSID_HIP(hipStreamSynchronize(cs));
        const int64_t ng = items_per_wave(K, TSID_BF16);
        for (int sd = 0; sd < 2; ++sd) d.plan[sd] = build_plan(c, hsp[sd], rows[sd], choose_E(d.sparse_nnz), ng);
        d.ready = true;
    } catch (...) {
        cleanup();
        free_dense(c, d);
        throw;
    }
    cleanup();
}

// Whether the current fit runs the dense head tiles: bf16 factors, k in
// {16, 32, 64, 128}, and either a forced tile fill (tsid_set_dense_tiles) or
// the default fill with at least a tenth of the cells in dense tiles.  The
// default is 0.15, and 0.10 at k = 128: there a sparse cell gathers a whole
// 256-byte row, which a tile shares among its 16 owner rows, so tiles pay
// off at a lower fill (measured sweeps: Rating-shaped, k = 64, fastest at
// 0.15 to 0.25; Billion-scale, k = 128, about 1% faster at 0.10 than 0.15).
#ifndef TSID_DENSE_FILL
#define TSID_DENSE_FILL 0.15f
#endif
#ifndef TSID_DENSE_FILL_K128
#define TSID_DENSE_FILL_K128 0.10f
#endif
#ifndef TSID_DENSE_MIN_SHARE
#define TSID_DENSE_MIN_SHARE 0.10
#endif
void ensure_dense(tsid_ctx *c, int prec) {
    Template &t = *c->tpl;
    const float mode = c->dense_fill;
    t.dense_use = false;
    if (mode == 0.f) return;
    if (!dense_supported(t.k, prec)) {
        if (mode > 0.f) fail(TSID_E_INVAL, "dense tiles need bf16 factors and k in {16, 32, 64, 128}");
        return;
    }
    const float fill = mode > 0.f ? mode : (t.k >= 128 ? TSID_DENSE_FILL_K128 : TSID_DENSE_FILL);
    if (!t.dense.ready || t.dense.fill != fill) {
        build_dense(c, fill);
        free_blocks(c, t.qb);  // the row blocks index the other cells' stream, which changed
    }
    t.dense_use = mode > 0.f ? true : t.dense.cells >= TSID_DENSE_MIN_SHARE * (double)t.nnz && t.dense.tiles > 0;
}

// Mini-batch streams and pointers for the context's batch count and seed
// (rebuilt when either changes), then the batch plans of precision prec.
void ensure_minibatch(tsid_ctx *c, int prec) {
    Template &t = *c->tpl;
    MiniPlan &mb = t.mb;
    const int32_t B = c->mb_batches;
    if (!mb.ready || mb.B != B || mb.seed != c->mb_seed) {
        free_minibatch(c, mb);
        for (int sd = 0; sd < 2; ++sd)
            if ((int64_t)B * (sd ? t.n_t : t.m_t) >= INT32_MAX)
                fail(TSID_E_INVAL, "n_batches times the template's rows (or columns) must be below 2^31");
        Arena &A = c->arena;
        hipStream_t cs = c->comp;
        const int64_t n = t.nnz;
        uint64_t *keys = nullptr, *keys_alt = nullptr;
        uint32_t *vals = nullptr, *vals_alt = nullptr, *tmp = nullptr;
        auto cleanup = [&]() {
            (void)hipStreamSynchronize(cs);
            A.release(keys);
            A.release(keys_alt);
            A.release(vals);
            A.release(vals_alt);
            A.release(tmp);
        };
        try {
            keys = A.alloc<uint64_t>(n);
            keys_alt = A.alloc<uint64_t>(n);
            vals = A.alloc<uint32_t>(n);
            vals_alt = A.alloc<uint32_t>(n);
            tmp = A.alloc<uint32_t>((int64_t)radix_scratch_elems(n));
            for (int sd = 0; sd < 2; ++sd) {
                const int32_t rows = sd ? t.n_t : t.m_t;
                const int64_t nkeys = (int64_t)B * rows;
                const int2 *st = sd ? t.stream_c : t.stream_r;
                batch_keys(st, sd ? t.col_ptr : t.row_ptr, rows, sd, c->mb_seed, B, keys, vals, cs);
                // stable: each batch keeps its cells bucketed by owner row in stream order
                const bool alt = radix_sort(keys, vals, keys_alt, vals_alt, n, bits_for(nkeys), tmp, cs);
                mb.stream[sd] = A.alloc<int2>(n);
                mb.ptr[sd] = A.alloc<int64_t>(nkeys + 1);
                gather_stream(st, alt ? vals_alt : vals, n, mb.stream[sd], cs);
                ptr_from_keys(alt ? keys_alt : keys, n, (int32_t)nkeys, 0, mb.ptr[sd], cs);
                mb.hptr[sd].resize((size_t)nkeys + 1);
                TSID_HIP(hipMemcpyAsync(mb.hptr[sd].data(), mb.ptr[sd], ((size_t)nkeys + 1) * 8,
                                        hipMemcpyDeviceToHost, cs));
                TSID_HIP(hipStreamSynchronize(cs));
            }
        } catch (...) {
            cleanup();
            free_minibatch(c, mb);
            throw;
        }
        cleanup();
        mb.B = B;
        mb.seed = c->mb_seed;
        mb.ready = true;
    }
    if (mb.plan[0][prec].empty()) {
        // items sized for a batch's share of the cells
        const int64_t E = choose_E(std::max<int64_t>(1, t.nnz / B), TSID_MB_TARGET_ITEMS);
        const int ng = items_per_wave(t.k, prec);
        int64_t most = 0;
        try {
            for (int sd = 0; sd < 2; ++sd) {
                const int32_t rows = sd ? t.n_t : t.m_t;
                auto &v = mb.plan[sd][prec];
                for (int32_t b = 0; b < B; ++b) {
                    const std::vector<int64_t> sub(mb.hptr[sd].begin() + (int64_t)b * rows,
                                                   mb.hptr[sd].begin() + (int64_t)b * rows + rows + 1);
                    v.push_back(build_plan(c, sub, rows, E, ng));
                    most = std::max<int64_t>(most, v.back().n_items);
                }
            }
        } catch (...) {
            for (int sd = 0; sd < 2; ++sd) {
                for (Plan &pl : mb.plan[sd][prec]) free_plan(c, pl);
                mb.plan[sd][prec].clear();
            }
            throw;
        }
        mb.max_items[prec] = most;
    }
}

// dense: whether a fit is about to run (the loss evaluation uses no tiles);
// extra_items: the largest work plan of a mini-batch fit (0 otherwise)
// item_only: the fit runs the item pass on both sides (no slab pass)
void ensure_fit_buffers(tsid_ctx *c, int32_t prec, int32_t epochs, bool dense, int64_t extra_items = 0,
                        bool item_only = false) {
    Template &t = *c->tpl;
    FitBufs &f = c->fb;
    Arena &A = c->arena;
    const int64_t lp = (int64_t)t.m_t * t.k, lq = (int64_t)t.n_t * t.k;
    ensure_plan(c, 0, prec);
    ensure_plan(c, 1, prec);
    if (item_only) {
        t.slab[0].use = t.slab[1].use = false;
    } else {
        const bool w0 = slab_wanted(c, 0, prec), w1 = slab_wanted(c, 1, prec);
        ensure_slab(c, 0, w0, w0 + w1);
        ensure_slab(c, 1, w1, w0 + w1);
    }
    if (dense)
        ensure_dense(c, prec);
    else
        t.dense_use = false;
    if (!f.P[0]) {
        for (int b = 0; b < 2; ++b) {
            f.P[b] = A.alloc<float>(lp);
            f.Q[b] = A.alloc<float>(lq);
        }
        f.normP = A.alloc<float>((int64_t)t.m_t * kLossRing);
        f.normQ = A.alloc<float>((int64_t)t.n_t * kLossRing);
        f.partial = A.alloc<double>((int64_t)reduce_scratch_elems(kLossRing));
    }
    const int64_t need = std::max({(int64_t)t.plan[0][prec].n_items, (int64_t)t.plan[1][prec].n_items,
                                   t.slab[0].use ? t.slab[0].lanes() : 0, t.slab[1].use ? t.slab[1].lanes() : 0,
                                   t.dense_use ? (int64_t)t.dense.plan[0].n_items + t.dense.n_segs[0] : 0,
                                   t.dense_use ? (int64_t)t.dense.plan[1].n_items : 0, extra_items});
    if (need > f.item_cap) {  // partial sums and per-item e^2, sized for this precision's plans
        A.release(f.carry_r);
        A.release(f.carry_c);
        A.release(f.e2);
        f.item_cap = 0;
        f.carry_r = A.alloc<float>(need * t.k);
        f.carry_c = A.alloc<float>(need * t.k);
        f.e2 = A.alloc<float>(need * kLossRing);
        f.item_cap = need;
    }
    if (prec == TSID_BF16 && !f.Pb[0]) {
        for (int b = 0; b < 2; ++b) {
            f.Pb[b] = A.alloc<uint16_t>(lp);
            f.Qb[b] = A.alloc<uint16_t>(lq);
        }
    }
    if (f.loss_cap < epochs + 1) {  // at least 4096 epochs, so that later fits rarely reallocate
        A.release(f.loss);
        const int32_t cap = std::max<int32_t>(epochs + 1, 4096);
        f.loss = A.alloc<double>(cap);
        f.loss_cap = cap;
    }
}

// Row blocks of the Q pass for this fit: automatic when the gathered P table
// exceeds TSID_QBLOCK_MIN_MB (blocks of about TSID_QBLOCK_MB of the table
// each, their count rounded up to a multiple of the XCDs, at most
// TSID_MAX_ROW_BLOCKS), else one.  More blocks raise the L2 hit rate of the
// gathers (Billion-scale: 53 % with 16, 76 % with 64) but cut the columns'
// runs shorter, and the per-run work (owner row, partial sum) then outweighs
// it; Billion-scale (256 MB of bf16 P) ran its Q pass in 5.02 ms with 16
// blocks, 4.89-4.93 with 24 and 5.11 with 32 (interleaved order below).
#ifndef TSID_QBLOCK_MB
#define TSID_QBLOCK_MB 11
#endif
#ifndef TSID_QBLOCK_MIN_MB
#define TSID_QBLOCK_MIN_MB 96
#endif
// XCDs of the device (gfx950: 8); the dispatcher hands consecutive
// workgroups to them in turn.
constexpr int kXcds = 8;

int32_t ensure_qblock(tsid_ctx *c, int prec) {
    Template &t = *c->tpl;
    BlockPlan &qb = t.qb;
    const int64_t table = (int64_t)t.m_t * t.k * (prec == TSID_BF16 ? 2 : 4);
    int32_t nb = c->row_blocks;
    if (nb == 0) {
        nb = 1;
        if (table > (int64_t)TSID_QBLOCK_MIN_MB << 20) {
            const int64_t want = (table + ((int64_t)TSID_QBLOCK_MB << 20) - 1) / ((int64_t)TSID_QBLOCK_MB << 20);
            nb = (int32_t)std::min<int64_t>((want + kXcds - 1) / kXcds * kXcds, TSID_MAX_ROW_BLOCKS);
        }
    }
    nb = (int32_t)std::min<int64_t>(nb, std::max<int32_t>(1, t.m_t));
    if (nb <= 1 || t.n_t == 0 || t.slab[1].use) return 1;
    const bool dn = t.dense_use && prec == TSID_BF16;
    Arena &A = c->arena;
    hipStream_t cs = c->comp;
    if (qb.nb != nb || qb.dense != dn) {
        free_blocks(c, qb);
        try {
            // the cells the Q pass walks, counted by their row (the P row it
            // gathers); block j starts at the first row with at least
            // j / nb of them before it
            std::vector<int64_t> rptr;
            if (dn) {
                rptr.resize((size_t)t.m_t + 1);
                TSID_HIP(hipMemcpy(rptr.data(), t.dense.sparse_ptr[0], rptr.size() * 8, hipMemcpyDeviceToHost));
            }
            const std::vector<int64_t> &rp = dn ? rptr : t.hptr[0];
            const int64_t total = rp[(size_t)t.m_t];
            qb.hrow_bounds.assign((size_t)nb + 1, (int64_t)t.m_t);
            qb.hrow_bounds[0] = 0;
            const bool equal_rows = std::getenv("TSID_QBLOCK_EQUAL_ROWS") != nullptr;  // tuning knob
            int64_t r = 0;
            for (int32_t j = 1; j < nb; ++j) {
                if (equal_rows || total == 0) {
                    qb.hrow_bounds[(size_t)j] = std::min<int64_t>((int64_t)j * ((t.m_t + nb - 1) / nb), t.m_t);
                    continue;
                }
                const int64_t target = (int64_t)(((__int128)j * total + nb - 1) / nb);
                while (r < t.m_t && rp[(size_t)r] - rp[0] < target) ++r;
                qb.hrow_bounds[(size_t)j] = r;
            }
            qb.row_bounds = A.alloc<int64_t>((int64_t)nb + 1);
            qb.bounds = A.alloc<int64_t>((int64_t)(nb + 1) * t.n_t);
            qb.part = A.alloc<float>((int64_t)nb * t.n_t * t.k);
            TSID_HIP(hipMemcpyAsync(qb.row_bounds, qb.hrow_bounds.data(), ((size_t)nb + 1) * 8, hipMemcpyHostToDevice,
                                    cs));
            launch_block_bounds(dn ? t.dense.sparse[1] : t.stream_c, dn ? t.dense.sparse_ptr[1] : t.col_ptr, t.n_t,
                                nb, qb.row_bounds, qb.bounds, cs);
            TSID_HIP(hipStreamSynchronize(cs));
        } catch (...) {
            free_blocks(c, qb);
            throw;
        }
        qb.nb = nb;
        qb.dense = dn;
    }
    BlockPlan::Combined &cb = qb.comb[prec];
    if (!cb.ready) {
        const int64_t n = (int64_t)(nb + 1) * t.n_t;
        std::vector<int64_t> hb((size_t)n);
        TSID_HIP(hipMemcpy(hb.data(), qb.bounds, (size_t)n * 8, hipMemcpyDeviceToHost));
        // Items sized for the blocks that run at one time (a group of kXcds):
        // enough of them to fill the device, each as long as that allows.
        // Billion-scale (24 blocks): 560 cells, Q pass 4.4 ms; sized per
        // block instead (80 cells, four times the waves) it took 4.9 ms, with
        // 160 / 320 / 640 / 1,280 / 2,560 cells 4.75 / 4.57 / 4.38 / 4.41 /
        // 4.45 ms.  Tuning knob TSID_QBLOCK_E: the cell count.
        const char *ee = std::getenv("TSID_QBLOCK_E");
        const int64_t pass_cells = dn ? t.dense.sparse_nnz : t.nnz;
        const int64_t E = ee && std::atoi(ee) > 0
                              ? (int64_t)std::atoi(ee)
                              : choose_E(std::max<int64_t>(1, pass_cells * std::min(nb, kXcds) / nb));
        const int ng = items_per_wave(t.k, prec), wg = items_per_workgroup(t.k, prec);
        const int64_t nv = (int64_t)nb * t.n_t;
        if (nv >= INT32_MAX) fail(TSID_E_INVAL, "too many row-block buckets");
        PlanLayout C;
        C.off.resize((size_t)nv + 1);
        C.endv.resize((size_t)nv + 1);
        C.E = E;
        std::vector<int64_t> base((size_t)nb), chunks((size_t)nb);
        int64_t cur = 0;
        for (int32_t j = 0; j < nb; ++j) {
            std::vector<int64_t> fake((size_t)t.n_t + 1, 0);  // prefix sums of the runs' lengths
            for (int32_t x = 0; x < t.n_t; ++x)
                fake[(size_t)x + 1] = fake[(size_t)x] + hb[(size_t)(j + 1) * t.n_t + x] - hb[(size_t)j * t.n_t + x];
            const PlanLayout L = layout_plan(fake, t.n_t, E, ng);
            const int64_t b0 = (cur + wg - 1) / wg * wg;  // every block starts a workgroup
            const int64_t nj = (int64_t)L.items.size();
            if (b0 + nj >= INT32_MAX) fail(TSID_E_INVAL, "row-block work plan too large");
            C.items.resize((size_t)(b0 + nj), -1);
            for (int64_t it = 0; it < nj; ++it)
                if (L.items[(size_t)it] >= 0) C.items[(size_t)(b0 + it)] = (int32_t)((int64_t)j * t.n_t + L.items[(size_t)it]);
            for (int32_t x = 0; x < t.n_t; ++x) {
                C.off[(size_t)j * t.n_t + x] = (uint32_t)(b0 + L.off[(size_t)x]);
                C.endv[(size_t)j * t.n_t + x] = (uint32_t)(b0 + L.endv[(size_t)x]);
            }
            C.spans = C.spans || L.spans;
            base[(size_t)j] = b0;
            chunks[(size_t)j] = (nj + wg - 1) / wg;
            cur = b0 + nj;
        }
        C.off[(size_t)nv] = C.endv[(size_t)nv] = (uint32_t)cur;
        // workgroup schedule: the blocks in groups of kXcds; in a group,
        // workgroup w takes the next chunk of the group's block w % kXcds.
        // order[]: the blocks in schedule order, taken alternately from both
        // ends (0, nb - 1, 1, nb - 2, ...), so that a group holds hot blocks
        // (few rows: the most observed) and cold ones (many rows) and the
        // rows the XCDs gather from at one time are about the same share of
        // the table in every group.  With consecutive blocks (tuning knob
        // TSID_QBLOCK_ORDER=0) the group of cold blocks spans most of the
        // table at once, more than the memory-side cache holds, and the
        // Billion-scale Q pass ran 5.47 ms instead of 5.02 (16 blocks).
        std::vector<int32_t> order((size_t)nb);
        const char *oe = std::getenv("TSID_QBLOCK_ORDER");
        const int omode = oe ? std::atoi(oe) : 1;
        for (int32_t q = 0; q < nb; ++q)
            order[(size_t)q] = omode == 1 ? ((q & 1) ? nb - 1 - q / 2 : q / 2) : q;
        std::vector<int32_t> sched;
        for (int32_t g0 = 0; g0 < nb; g0 += kXcds) {
            int64_t most = 0;
            for (int32_t q = g0; q < std::min(nb, g0 + kXcds); ++q)
                most = std::max(most, chunks[(size_t)order[(size_t)q]]);
            for (int64_t ch = 0; ch < most; ++ch)
                for (int x = 0; x < kXcds; ++x) {
                    const int32_t q = g0 + x;
                    const int32_t j = q < nb ? order[(size_t)q] : -1;
                    sched.push_back(j >= 0 && ch < chunks[(size_t)j] ? (int32_t)(base[(size_t)j] / wg + ch) : -1);
                }
        }
        try {
            cb.plan = upload_plan(c, C, (int32_t)nv);
            cb.sched = A.alloc<int32_t>((int64_t)sched.size());
            TSID_HIP(hipMemcpy(cb.sched, sched.data(), sched.size() * 4, hipMemcpyHostToDevice));
            cb.n_wg = (int64_t)sched.size();
            cb.carry = A.alloc<float>((cur / ng + 1) * t.k);
        } catch (...) {
            free_plan(c, cb.plan);
            A.release(cb.sched);
            A.release(cb.carry);
            cb = BlockPlan::Combined{};
            throw;
        }
        cb.ready = true;
    }
    return nb;
}

PassArgs pass_args(const Template &t, int side, const tsid_fit_opts &o, int32_t *err) {
    PassArgs a{};
    // with dense head tiles the item pass walks the other cells only
    const bool dn = t.dense_use && o.prec == TSID_BF16;
    const Plan &pl = dn ? t.dense.plan[side] : t.plan[side][o.prec];
    a.stream = dn ? t.dense.sparse[side] : (side ? t.stream_c : t.stream_r);
    a.ptr = dn ? t.dense.sparse_ptr[side] : (side ? t.col_ptr : t.row_ptr);
    a.dptr = dn ? (side ? t.col_ptr : t.row_ptr) : nullptr;
    a.gd = dn ? t.dense.gd[side] : nullptr;
    a.gd_tile_ptr = dn ? t.dense.tile_ptr[side] : nullptr;
    a.items = pl.items;
    a.item_off = pl.item_off;
    a.item_end = pl.item_end;
    a.n_items_dev = nullptr;
    a.n_items = pl.n_items;
    a.rows = side ? t.n_t : t.m_t;
    a.y_rows = side ? t.m_t : t.n_t;
    a.E = pl.E;
    a.lam = o.lambda;
    a.lr = o.lr;
    a.xi = o.clip_xi;
    a.clip = o.clip;
    a.degree = side_scaled(o.step, side);
    a.err = err;
    return a;
}

DenseArgs dense_args(const Template &t, int side, int32_t *err) {
    DenseArgs a{};
    const DensePlan &d = t.dense;
    a.rows = side ? t.n_t : t.m_t;
    a.y_rows = side ? t.m_t : t.n_t;
    a.n_segs = d.n_segs[side];
    a.seg_tile = d.seg_tile[side];
    a.seg_order = d.seg_order[side];
    a.seg_stripe = d.seg_stripe[side];
    a.stripe_seg = d.stripe_seg[side];
    a.tile_other = d.tile_other[side];
    a.R = d.R[side];
    a.gd = d.gd[side];
    a.part = d.part[side];
    a.multi = d.multi[side];
    a.n_multi = d.n_multi[side];
    a.err = err;
    return a;
}

SlabArgs slab_args(const Template &t, int side, const tsid_fit_opts &o, int32_t *err) {
    const SlabPlan &sp = t.slab[side];
    SlabArgs a{};
    a.sblk = sp.sblk;
    a.seg = sp.seg;
    a.ptr = side ? t.col_ptr : t.row_ptr;
    a.rows = side ? t.n_t : t.m_t;
    a.y_rows = side ? t.m_t : t.n_t;
    a.C = sp.C;
    a.n_slabs = sp.n_slabs;
    a.slabs_per_unit = sp.S;
    a.units_per_block = sp.U;
    a.carry = sp.carry;
    a.lam = o.lambda;
    a.lr = o.lr;
    a.xi = o.clip_xi;
    a.clip = o.clip;
    a.degree = side_scaled(o.step, side);
    a.err = err;
    return a;
}

// S of the multi-view term: validated on the host (ids inside the template's
// columns, values finite and >= 0, no repeated entry, symmetric with equal
// values both ways), then stored as CSR in input order within each row.
void set_similarity(tsid_ctx *c, const int32_t *row, const int32_t *col, const float *val, int64_t nnz,
                    float beta) {
    if (!c->tpl) fail(TSID_E_STATE, "no template: call tsid_build_template first");
    Template &t = *c->tpl;
    if (nnz < 0) fail(TSID_E_INVAL, "nnz < 0");
    if (nnz > 0 && (!row || !col || !val)) fail(TSID_E_INVAL, "NULL similarity arrays");
    if (!(beta >= 0.f) || !std::isfinite(beta)) fail(TSID_E_INVAL, "beta must be finite and >= 0");
    std::vector<std::pair<uint64_t, uint32_t>> fw((size_t)nnz), bw((size_t)nnz);
    for (int64_t e = 0; e < nnz; ++e) {
        if (row[e] < 0 || row[e] >= t.n_t || col[e] < 0 || col[e] >= t.n_t)
            fail(TSID_E_RANGE, "similarity id outside the template's columns");
        if (!(val[e] >= 0.f) || !std::isfinite(val[e])) fail(TSID_E_INVAL, "similarity values must be finite and >= 0");
        uint32_t bits;
        std::memcpy(&bits, &val[e], 4);
        fw[(size_t)e] = {((uint64_t)(uint32_t)row[e] << 32) | (uint32_t)col[e], bits};
        bw[(size_t)e] = {((uint64_t)(uint32_t)col[e] << 32) | (uint32_t)row[e], bits};
    }
    std::sort(fw.begin(), fw.end());
    std::sort(bw.begin(), bw.end());
    for (size_t e = 1; e < fw.size(); ++e)
        if (fw[e].first == fw[e - 1].first) fail(TSID_E_DUP, "repeated similarity entry");
    if (fw != bw) fail(TSID_E_INVAL, "the similarity matrix must be symmetric");
    free_sim(c, t.sim);
    if (nnz == 0 || beta == 0.f) return;  // the term is off
    std::vector<int64_t> ptr((size_t)t.n_t + 1, 0);
    for (int64_t e = 0; e < nnz; ++e) ptr[(size_t)row[e] + 1] += 1;
    for (int32_t x = 0; x < t.n_t; ++x) ptr[(size_t)x + 1] += ptr[(size_t)x];
    std::vector<int64_t> fill(ptr.begin(), ptr.end() - 1);
    std::vector<int32_t> hc((size_t)nnz);
    std::vector<float> hv((size_t)nnz);
    for (int64_t e = 0; e < nnz; ++e) {
        const int64_t at = fill[(size_t)row[e]]++;
        hc[(size_t)at] = col[e];
        hv[(size_t)at] = val[e];
    }
    SimPlan sp;
    Arena &A = c->arena;
    hipStream_t cs = c->comp;
    try {
        sp.ptr = A.alloc<int64_t>((int64_t)t.n_t + 1);
        sp.col = A.alloc<int32_t>(nnz);
        sp.val = A.alloc<float>(nnz);
        sp.gs = A.alloc<float>((int64_t)t.n_t * t.k);
        sp.se = A.alloc<float>((int64_t)t.n_t * kLossRing);
        TSID_HIP(hipMemcpyAsync(sp.ptr, ptr.data(), ptr.size() * 8, hipMemcpyHostToDevice, cs));
        TSID_HIP(hipMemcpyAsync(sp.col, hc.data(), (size_t)nnz * 4, hipMemcpyHostToDevice, cs));
        TSID_HIP(hipMemcpyAsync(sp.val, hv.data(), (size_t)nnz * 4, hipMemcpyHostToDevice, cs));
        TSID_HIP(hipStreamSynchronize(cs));  // the host vectors go out of scope
    } catch (...) {
        free_sim(c, sp);
        throw;
    }
    sp.on = true;
    sp.beta = beta;
    sp.nnz = nnz;
    t.sim = sp;
}

// Mini-batch epochs: epoch ep takes one step per batch beta (global step
// s = ep * B + beta), each an item pass of both sides over the batch's cells
// from the factors the previous step left (P and Q of one step both move
// from the same iterate, as in a Jacobi epoch); lines without a cell in the
// batch keep their rows.  The loss of epoch ep is evaluated over every cell
// before its first step.  The factor buffers alternate every step, so the
// iterate before step s sits in buffer s & 1.
void fit_minibatch(tsid_ctx *c, float *P, float *Q, const tsid_fit_opts *o, double *loss_hist) {
    Template &t = *c->tpl;
    if (c->pass_kernel == TSID_PASS_SLAB)
        fail(TSID_E_INVAL, "mini-batch epochs run the item pass (the slab pass walks whole buckets)");
    if (c->dense_fill > 0.f) fail(TSID_E_INVAL, "mini-batch epochs do not use dense tiles");
    const int32_t B = c->mb_batches;
    if ((int64_t)o->epochs * B >= INT32_MAX - 1) fail(TSID_E_INVAL, "epochs times n_batches must be below 2^31 - 1");
    const int K = t.k, prec = o->prec, T = o->epochs;
    ensure_minibatch(c, prec);
    MiniPlan &mb = t.mb;
    // the steps walk the batch streams; with bf16 factors the epochs' loss
    // passes may still take the dense head tiles (automatic rule)
    ensure_fit_buffers(c, prec, T, true, mb.max_items[prec], true);
    const bool dn = t.dense_use && prec == TSID_BF16;
    c->epochs_done = 0;
    c->dense_used = tsid_dense_info{};
    c->used_kernel[0] = c->used_kernel[1] = TSID_PASS_ITEM;
    c->used_blocks = 1;
    FitBufs &f = c->fb;
    hipStream_t cs = c->comp;
    const int64_t lp = (int64_t)t.m_t * K, lq = (int64_t)t.n_t * K;
    if (lp) TSID_HIP(hipMemcpyAsync(f.P[0], P, (size_t)lp * 4, hipMemcpyDeviceToDevice, cs));
    if (lq) TSID_HIP(hipMemcpyAsync(f.Q[0], Q, (size_t)lq * 4, hipMemcpyDeviceToDevice, cs));
    if (prec == TSID_BF16) {
        launch_to_bf16(f.P[0], lp, f.Pb[0], cs);
        launch_to_bf16(f.Q[0], lq, f.Qb[0], cs);
    }
    TSID_HIP(hipMemsetAsync(c->err_dev, 0, ERR_SLOTS * sizeof(int32_t), cs));
    // the loss pass walks the whole stream with the template's own plan (with
    // dense tiles: the tiles' loss-only kernel plus the item pass over the
    // other cells, as in a Jacobi epoch)
    PassArgs full = pass_args(t, 0, *o, c->err_dev);
    full.skip_after_nonfinite = 1;
    full.Xn = nullptr;
    DenseArgs dfull = dense_args(t, 0, c->err_dev);
    dfull.skip_after_nonfinite = 1;
    const int64_t ne_items = full.n_items;
    const int64_t ne = ne_items + (dn ? dfull.n_segs : 0);
    PassArgs step[2] = {pass_args(t, 0, *o, c->err_dev), pass_args(t, 1, *o, c->err_dev)};
    for (int sd = 0; sd < 2; ++sd) {
        step[sd].dptr = nullptr;  // the batch streams hold every cell of the batch
        step[sd].gd = nullptr;
        step[sd].gd_tile_ptr = nullptr;
        step[sd].stream = mb.stream[sd];
        step[sd].keep_empty = 1;
        step[sd].skip_after_nonfinite = 1;
        step[sd].e2 = nullptr;
        step[sd].norm = nullptr;
    }
    step[0].carry = f.carry_r;
    step[1].carry = f.carry_c;
    if (c->timing) ensure_events(c, (size_t)T);
    const bool want_loss = loss_hist != nullptr;
    int pend = 0;
    auto flush = [&](int upto, std::pair<hipEvent_t, hipEvent_t> ev) {
        launch_loss_reduce(f.e2, f.item_cap, ne, f.normP, t.m_t, f.normQ, t.n_t, o->lambda, upto - pend,
                           f.partial, f.loss + pend, nullptr, pend, cs, ev.first, ev.second);
        pend = upto;
    };
    auto loss_pass = [&](int ep, int buf) {
        const int slot = ep % kLossRing;
        full.epoch = ep * B;  // skipped after a failure in an earlier step
        full.X = f.P[buf];
        full.Y = prec ? (const void *)f.Qb[buf] : (const void *)f.Q[buf];
        full.e2 = f.e2 + slot * f.item_cap;
        full.norm = f.normP + (int64_t)slot * t.m_t;
        if (dn && dfull.n_segs) {
            dfull.epoch = ep * B;
            dfull.X = f.Pb[buf];
            dfull.Y = f.Qb[buf];
            dfull.e2 = full.e2 + ne_items;
            launch_dense_pass(K, true, dfull, cs);
        }
        launch_item_pass(K, prec, true, full, cs);
        launch_row_norms(K, f.Q[buf], t.n_t, f.normQ + (int64_t)slot * t.n_t, cs);
    };
    int cur = 0;
    for (int ep = 0; ep < T; ++ep) {
        auto eve = timed(c, ep, TK_EPOCH);
        if (eve.first) TSID_HIP(hipEventRecord(eve.first, cs));
        if (want_loss) loss_pass(ep, cur);
        for (int32_t beta = 0; beta < B; ++beta) {
            const int nxt = cur ^ 1;
            for (int sd = 0; sd < 2; ++sd) {
                PassArgs &a = step[sd];
                const int32_t rows = sd ? t.n_t : t.m_t;
                const Plan &pl = mb.plan[sd][prec][(size_t)beta];
                a.ptr = mb.ptr[sd] + (int64_t)beta * rows;
                a.items = pl.items;
                a.item_off = pl.item_off;
                a.item_end = pl.item_end;
                a.n_items = pl.n_items;
                a.E = pl.E;
                a.epoch = ep * B + beta;
                float *const *X = sd ? f.Q : f.P;
                float *const *Y = sd ? f.P : f.Q;
                uint16_t *const *Xb = sd ? f.Qb : f.Pb;
                uint16_t *const *Yb = sd ? f.Pb : f.Qb;
                a.X = X[cur];
                a.Y = prec ? (const void *)Yb[cur] : (const void *)Y[cur];
                a.Xn = X[nxt];
                a.Xn_b = prec ? Xb[nxt] : nullptr;
                auto ev = beta == 0 ? timed(c, ep, sd ? TK_QPASS : TK_PPASS) : std::pair<hipEvent_t, hipEvent_t>{};
                launch_item_pass(K, prec, false, a, cs, ev.first, ev.second);
                if (pl.spans) {
                    ev = beta == 0 ? timed(c, ep, sd ? TK_QFIX : TK_PFIX) : std::pair<hipEvent_t, hipEvent_t>{};
                    launch_fixup(K, prec, a, cs, ev.first, ev.second);
                }
            }
            cur = nxt;
        }
        if (eve.second) TSID_HIP(hipEventRecord(eve.second, cs));
        if (want_loss && ep % kLossRing == kLossRing - 1) flush(ep + 1, timed(c, ep, TK_REDUCE));
    }
    if (want_loss) {  // L(P_T, Q_T), then the epochs not reduced yet
        loss_pass(T, cur);
        flush(T + 1, {nullptr, nullptr});
    }
    std::vector<double> hist((size_t)T + 1);
    if (loss_hist) TSID_HIP(hipMemcpyAsync(hist.data(), f.loss, (size_t)(T + 1) * 8, hipMemcpyDeviceToHost, cs));
    TSID_HIP(hipMemcpyAsync(c->err_host, c->err_dev, ERR_SLOTS * 4, hipMemcpyDeviceToHost, cs));
    TSID_HIP(hipStreamSynchronize(cs));
    if (c->timing) collect_timing(c, T);
    const int32_t bad = c->err_host[ERR_NONFINITE];
    // with a failure in step s: the iterate before it, and the whole epochs before it
    const int64_t s_fail = bad ? bad - 1 : (int64_t)T * B;
    const int last = bad ? (int)(s_fail / B) : T;
    c->epochs_done = last;
    const int src = (int)(s_fail & 1);
    if (lp) TSID_HIP(hipMemcpyAsync(P, f.P[src], (size_t)lp * 4, hipMemcpyDeviceToDevice, cs));
    if (lq) TSID_HIP(hipMemcpyAsync(Q, f.Q[src], (size_t)lq * 4, hipMemcpyDeviceToDevice, cs));
    TSID_HIP(hipStreamSynchronize(cs));
    if (loss_hist) {
        for (int ep = 0; ep <= T; ++ep) loss_hist[ep] = ep <= last ? hist[ep] : NAN;
    }
    if (bad)
        fail(TSID_E_NONFINITE, "non-finite update in epoch " + std::to_string(last) + ", batch " +
                                   std::to_string(s_fail % B));
}

void fit(tsid_ctx *c, float *P, float *Q, const tsid_fit_opts *o, double *loss_hist) {
    if (!c->tpl) fail(TSID_E_STATE, "no template: call tsid_build_template first");
    check_opts(o);
    Template &t = *c->tpl;
    if ((t.m_t && !P) || (t.n_t && !Q)) fail(TSID_E_INVAL, "NULL factor pointer");
    if (o->clip == 2) {  // per-entry terms: the item pass only
        if (c->pass_kernel == TSID_PASS_SLAB) fail(TSID_E_INVAL, "per-entry clipping runs the item pass");
        if (c->dense_fill > 0.f) fail(TSID_E_INVAL, "per-entry clipping does not use dense tiles");
    }
    const SimPlan &sim = t.sim;
    if (sim.on) {  // the similarity term joins the item pass's Q update
        if (o->clip == 2) fail(TSID_E_INVAL, "the similarity term has no per-entry form (clip 2)");
        if (c->mb_batches > 0) fail(TSID_E_INVAL, "the similarity term runs with full-gradient epochs only");
        if (c->pass_kernel == TSID_PASS_SLAB) fail(TSID_E_INVAL, "the similarity term runs on the item pass");
    }
    if (c->mb_batches > 0) return fit_minibatch(c, P, Q, o, loss_hist);
    ensure_fit_buffers(c, o->prec, o->epochs, o->clip != 2, 0, o->clip == 2 || sim.on);
    const int32_t nb = ensure_qblock(c, o->prec);  // row blocks of the Q pass (1: one pass)
    c->used_blocks = nb;
    c->epochs_done = 0;
    FitBufs &f = c->fb;
    hipStream_t cs = c->comp;
    const int K = t.k, prec = o->prec, T = o->epochs;
    const int64_t lp = (int64_t)t.m_t * K, lq = (int64_t)t.n_t * K;
    if (lp) TSID_HIP(hipMemcpyAsync(f.P[0], P, (size_t)lp * 4, hipMemcpyDeviceToDevice, cs));
    if (lq) TSID_HIP(hipMemcpyAsync(f.Q[0], Q, (size_t)lq * 4, hipMemcpyDeviceToDevice, cs));
    if (prec == TSID_BF16) {
        launch_to_bf16(f.P[0], lp, f.Pb[0], cs);
        launch_to_bf16(f.Q[0], lq, f.Qb[0], cs);
    }
    TSID_HIP(hipMemsetAsync(c->err_dev, 0, ERR_SLOTS * sizeof(int32_t), cs));
    PassArgs ar = pass_args(t, 0, *o, c->err_dev), ac = pass_args(t, 1, *o, c->err_dev);
    ar.skip_after_nonfinite = ac.skip_after_nonfinite = 1;
    if (sim.on) {
        ac.gx = sim.gs;
        ac.gx_scale = 2.0f * sim.beta;
    }
    SlabArgs sr = slab_args(t, 0, *o, c->err_dev), sc = slab_args(t, 1, *o, c->err_dev);
    sr.skip_after_nonfinite = sc.skip_after_nonfinite = 1;
    const SlabPlan &sp_r = t.slab[0], &sp_c = t.slab[1];
    // Slab passes on both sides run as one launch per epoch (and their
    // finishes as another): the Q pass reads only the old factors.
    const bool slab_pair = sp_r.use && sp_c.use && !sim.on;
    // Likewise the item passes (after both sides' dense-tile launches), unless
    // the Q pass runs in row blocks.
    const bool item_pair = !sp_r.use && !sp_c.use && nb <= 1;
    // Both sides' dense-tile launches are one grid whenever both passes are
    // item passes (the Q side reads only the old factors' bf16 copies), also
    // when the Q pass runs in row blocks.
    const bool dn = t.dense_use && prec == TSID_BF16;
    const bool dense_pair = dn && !sp_r.use && !sp_c.use;
    DenseArgs dr = dense_args(t, 0, c->err_dev), dc = dense_args(t, 1, c->err_dev);
    dr.skip_after_nonfinite = dc.skip_after_nonfinite = 1;
    c->dense_used = tsid_dense_info{};
    if (dn) c->dense_used = tsid_dense_info{t.dense.cells, t.dense.tiles, {t.dense.stripes[0], t.dense.stripes[1]}};
    c->used_kernel[0] = sp_r.use ? TSID_PASS_SLAB : TSID_PASS_ITEM;
    c->used_kernel[1] = sp_c.use ? TSID_PASS_SLAB : TSID_PASS_ITEM;
    if (c->timing) ensure_events(c, (size_t)T);
    // Loss terms of epoch ep go to ring slot ep % kLossRing; a full ring (and
    // the end of the fit) is reduced in one batch into f.loss.
    const bool want_loss = loss_hist != nullptr;
    // loss terms per epoch: one per item of the P pass (or per lane of the
    // slab pass), then with dense tiles one per work segment
    const int64_t ne_items = sp_r.use ? sp_r.lanes() : (int64_t)ar.n_items;
    const int64_t ne = ne_items + (dn ? dr.n_segs : 0);
    int pend = 0;  // first epoch whose loss is not reduced yet
    auto flush = [&](int upto, std::pair<hipEvent_t, hipEvent_t> ev) {
        launch_loss_reduce(f.e2, f.item_cap, ne, f.normP, t.m_t, f.normQ, t.n_t, o->lambda, upto - pend,
                           f.partial, f.loss + pend, c->err_dev, pend, cs, ev.first, ev.second,
                           sim.on ? sim.se : nullptr, t.n_t, 0.5 * (double)sim.beta);
        pend = upto;
    };
    for (int ep = 0; ep < T; ++ep) {
        const int cur = ep & 1, nxt = cur ^ 1, slot = ep % kLossRing;
        // P pass (CSR): owner P_t, gathered Q_t
        float *e2 = want_loss ? f.e2 + slot * f.item_cap : nullptr;
        float *normp = want_loss ? f.normP + (int64_t)slot * t.m_t : nullptr;
        float *normq = want_loss ? f.normQ + (int64_t)slot * t.n_t : nullptr;
        auto ev = timed(c, ep, TK_PPASS);
        if (sp_r.use) {
            sr.epoch = ep;
            sr.X = f.P[cur];
            sr.Y = f.Q[cur];
            sr.Xn = f.P[nxt];
            sr.e2 = e2;
            sr.norm = normp;
            if (slab_pair) {
                sc.epoch = ep;
                sc.X = f.Q[cur];
                sc.Y = f.P[cur];
                sc.Xn = f.Q[nxt];
                sc.e2 = nullptr;
                sc.norm = normq;
                launch_slab_pass_pair(K, sr, sp_r.units(), sc, sp_c.units(), cs, ev.first, ev.second);
                if (sp_r.U > 1 && sp_c.U > 1) {
                    ev = timed(c, ep, TK_PFIX);
                    launch_slab_finish_pair(K, sr, sc, cs, ev.first, ev.second);
                } else if (sp_r.U > 1 || sp_c.U > 1) {
                    ev = timed(c, ep, TK_PFIX);
                    launch_slab_finish(K, sp_r.U > 1 ? sr : sc, cs, ev.first, ev.second);
                }
            } else {
                launch_slab_pass(K, false, sr, sp_r.units(), cs, ev.first, ev.second);
                if (sp_r.U > 1) {
                    ev = timed(c, ep, TK_PFIX);
                    launch_slab_finish(K, sr, cs, ev.first, ev.second);
                }
            }
        } else {
            if (dense_pair && (dr.n_segs || dc.n_segs)) {  // both sides' tiles in one launch
                dr.epoch = dc.epoch = ep;
                dr.X = f.Pb[cur];
                dr.Y = f.Qb[cur];
                dr.e2 = e2 ? e2 + ne_items : nullptr;
                dc.X = f.Qb[cur];
                dc.Y = f.Pb[cur];
                dc.e2 = nullptr;
                auto evd = timed(c, ep, TK_PDENSE);
                launch_dense_pass_pair(K, dr, dc, cs, evd.first, evd.second);
            } else if (dn && dr.n_segs) {
                dr.epoch = ep;
                dr.X = f.Pb[cur];
                dr.Y = f.Qb[cur];
                dr.e2 = e2 ? e2 + ne_items : nullptr;
                auto evd = timed(c, ep, TK_PDENSE);
                launch_dense_pass(K, false, dr, cs, evd.first, evd.second);
            }
            ar.epoch = ep;
            ar.X = f.P[cur];
            ar.Y = prec ? (const void *)f.Qb[cur] : (const void *)f.Q[cur];
            ar.Xn = f.P[nxt];
            ar.Xn_b = prec ? f.Pb[nxt] : nullptr;
            ar.carry = f.carry_r;
            ar.e2 = e2;
            ar.norm = normp;
            if (!item_pair) {  // else launched with the Q pass
                launch_item_pass(K, prec, false, ar, cs, ev.first, ev.second);
                if ((dn ? t.dense.plan[0] : t.plan[0][prec]).spans) {
                    ev = timed(c, ep, TK_PFIX);
                    launch_fixup(K, prec, ar, cs, ev.first, ev.second);
                }
            }
        }
        const auto ev_p = ev;
        // Q pass (CSC): owner Q_t, gathered P_t (the old P: a simultaneous step)
        if (sim.on)  // the similarity sums at Q_t, added to the Q gradients
            launch_sim_terms(K, sim.ptr, sim.col, sim.val, t.n_t, f.Q[cur], sim.gs,
                             want_loss ? sim.se + (int64_t)slot * t.n_t : nullptr, cs);
        ev = slab_pair || item_pair ? std::pair<hipEvent_t, hipEvent_t>{} : timed(c, ep, TK_QPASS);
        if (slab_pair) {
            // launched with the P pass
        } else if (sp_c.use) {
            sc.epoch = ep;
            sc.X = f.Q[cur];
            sc.Y = f.P[cur];
            sc.Xn = f.Q[nxt];
            sc.e2 = nullptr;
            sc.norm = normq;
            launch_slab_pass(K, false, sc, sp_c.units(), cs, ev.first, ev.second);
            if (sp_c.U > 1) {
                ev = timed(c, ep, TK_QFIX);
                launch_slab_finish(K, sc, cs, ev.first, ev.second);
            }
        } else {
            if (dn && dc.n_segs && !dense_pair) {
                dc.epoch = ep;
                dc.X = f.Qb[cur];
                dc.Y = f.Pb[cur];
                dc.e2 = nullptr;
                auto evd = timed(c, ep, TK_QDENSE);
                launch_dense_pass(K, false, dc, cs, evd.first, evd.second);
            }
            ac.epoch = ep;
            ac.X = f.Q[cur];
            ac.Y = prec ? (const void *)f.Pb[cur] : (const void *)f.P[cur];
            ac.Xn = f.Q[nxt];
            ac.Xn_b = prec ? f.Qb[nxt] : nullptr;
            ac.carry = f.carry_c;
            ac.e2 = nullptr;
            ac.norm = normq;
            if (nb > 1) {
                // every row block in one launch, each XCD on its own block of
                // P at a time, each (block, column) run leaving its partial
                // sum; then the combine kernel adds them in block order and
                // updates Q
                const BlockPlan::Combined &cb = t.qb.comb[prec];
                PassArgs bj = ac;
                bj.ptr = t.qb.bounds;
                bj.ptr_end = t.qb.bounds + t.n_t;
                bj.rows = (int32_t)((int64_t)nb * t.n_t);
                bj.owner_mod = t.n_t;
                bj.items = cb.plan.items;
                bj.item_off = cb.plan.item_off;
                bj.item_end = cb.plan.item_end;
                bj.n_items = cb.plan.n_items;
                bj.E = cb.plan.E;
                bj.carry = cb.carry;
                bj.carry_per_wave = 1;
                bj.norm = nullptr;
                bj.partial_out = t.qb.part;
                launch_item_pass_sched(K, prec, bj, cb.sched, cb.n_wg, cs, ev.first, ev.second);
                // the fixup of runs longer than a wave and the combine are
                // timed as the Q pass's fixups
                ev = timed(c, ep, TK_QFIX);
                if (cb.plan.spans) launch_fixup(K, prec, bj, cs, ev.first, nullptr);
                launch_block_combine(K, prec, ac, t.qb.part, nb, cs, cb.plan.spans ? nullptr : ev.first, ev.second);
            } else if (item_pair) {
                launch_item_pass_pair(K, prec, ar, ac, cs, ev_p.first, ev_p.second);
                if ((dn ? t.dense.plan[0] : t.plan[0][prec]).spans) {
                    ev = timed(c, ep, TK_PFIX);
                    launch_fixup(K, prec, ar, cs, ev.first, ev.second);
                }
                if ((dn ? t.dense.plan[1] : t.plan[1][prec]).spans) {
                    ev = timed(c, ep, TK_QFIX);
                    launch_fixup(K, prec, ac, cs, ev.first, ev.second);
                }
            } else {
                launch_item_pass(K, prec, false, ac, cs, ev.first, ev.second);
                if ((dn ? t.dense.plan[1] : t.plan[1][prec]).spans) {
                    ev = timed(c, ep, TK_QFIX);
                    launch_fixup(K, prec, ac, cs, ev.first, ev.second);
                }
            }
        }
        if (want_loss && slot == kLossRing - 1) flush(ep + 1, timed(c, ep, TK_REDUCE));
    }
    const int fin = T & 1;
    if (want_loss) {  // L(P_T, Q_T), then the epochs not reduced yet
        const int slot = T % kLossRing;
        if (sp_r.use) {
            sr.epoch = T;
            sr.X = f.P[fin];
            sr.Y = f.Q[fin];
            sr.Xn = nullptr;
            sr.e2 = f.e2 + slot * f.item_cap;
            sr.norm = f.normP + (int64_t)slot * t.m_t;
            launch_slab_pass(K, true, sr, sp_r.units(), cs);
        } else {
            if (dn && dr.n_segs) {
                dr.epoch = T;
                dr.X = f.Pb[fin];
                dr.Y = f.Qb[fin];
                dr.e2 = f.e2 + slot * f.item_cap + ne_items;
                launch_dense_pass(K, true, dr, cs);
            }
            ar.epoch = T;
            ar.X = f.P[fin];
            ar.Y = prec ? (const void *)f.Qb[fin] : (const void *)f.Q[fin];
            ar.Xn = nullptr;
            ar.e2 = f.e2 + slot * f.item_cap;
            ar.norm = f.normP + (int64_t)slot * t.m_t;
            launch_item_pass(K, prec, true, ar, cs);
        }
        launch_row_norms(K, f.Q[fin], t.n_t, f.normQ + (int64_t)slot * t.n_t, cs);
        if (sim.on)
            launch_sim_terms(K, sim.ptr, sim.col, sim.val, t.n_t, f.Q[fin], sim.gs, sim.se + (int64_t)slot * t.n_t,
                             cs);
        flush(T + 1, {nullptr, nullptr});
    }
    std::vector<double> hist((size_t)T + 1);
    if (loss_hist) TSID_HIP(hipMemcpyAsync(hist.data(), f.loss, (size_t)(T + 1) * 8, hipMemcpyDeviceToHost, cs));
    TSID_HIP(hipMemcpyAsync(c->err_host, c->err_dev, ERR_SLOTS * 4, hipMemcpyDeviceToHost, cs));
    TSID_HIP(hipStreamSynchronize(cs));
    if (c->timing) collect_timing(c, T);
    const int32_t bad = c->err_host[ERR_NONFINITE];
    const int last = bad ? bad - 1 : T;  // factors to return: (P_last, Q_last)
    c->epochs_done = last;
    const int src = last & 1;
    if (lp) TSID_HIP(hipMemcpyAsync(P, f.P[src], (size_t)lp * 4, hipMemcpyDeviceToDevice, cs));
    if (lq) TSID_HIP(hipMemcpyAsync(Q, f.Q[src], (size_t)lq * 4, hipMemcpyDeviceToDevice, cs));
    TSID_HIP(hipStreamSynchronize(cs));
    if (loss_hist) {
        for (int ep = 0; ep <= T; ++ep) loss_hist[ep] = ep <= last ? hist[ep] : NAN;
    }
    if (bad) fail(TSID_E_NONFINITE, "non-finite update in epoch " + std::to_string(bad - 1));
}

void loss(tsid_ctx *c, const float *P, const float *Q, float lambda, double *out) {
    if (!c->tpl) fail(TSID_E_STATE, "no template");
    Template &t = *c->tpl;
    if (!out) fail(TSID_E_INVAL, "out is NULL");
    if ((t.m_t && !P) || (t.n_t && !Q)) fail(TSID_E_INVAL, "NULL factor pointer");
    if (!(lambda >= 0.f) || !std::isfinite(lambda)) fail(TSID_E_INVAL, "lambda must be finite and >= 0");
    check_aligned(P, "P");
    check_aligned(Q, "Q");
    ensure_fit_buffers(c, TSID_FP32, 0, false);
    FitBufs &f = c->fb;
    hipStream_t cs = c->comp;
    tsid_fit_opts o{0, lambda, 1.f, 1.f, 0, TSID_FP32, TSID_STEP_SUM};
    PassArgs a = pass_args(t, 0, o, c->err_dev);
    a.X = P;
    a.Y = Q;
    a.e2 = f.e2;
    a.norm = f.normP;
    a.epoch = 0;
    a.skip_after_nonfinite = 0;
    launch_item_pass(t.k, TSID_FP32, true, a, cs);
    launch_row_norms(t.k, Q, t.n_t, f.normQ, cs);
    launch_loss_reduce(f.e2, f.item_cap, t.plan[0][TSID_FP32].n_items, f.normP, t.m_t, f.normQ, t.n_t,
                       lambda, 1, f.partial, f.loss, nullptr, -1, cs);
    TSID_HIP(hipMemcpyAsync(out, f.loss, 8, hipMemcpyDeviceToHost, cs));
    TSID_HIP(hipStreamSynchronize(cs));
}

// ------------------------------------------------ allocation-free loss

// Device scratch of tsid_loss_noalloc: one array per device, placed by the
// code object loader, never allocated by the library.  In host code the name
// is a host-side stand-in; the device address comes from
// hipGetSymbolAddress, once per device (noalloc_scratch_on), and only that
// address is handed to kernels and copies.
constexpr size_t kNoAllocBytes = TSID_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch array (looked up with the device
// current, at context creation).
void *noalloc_scratch_on(int device) {
    if (device < 0 || device >= kMaxDevices) fail(TSID_E_DEVICE, "device id beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *ptr = nullptr;
        TSID_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
        if (!ptr) fail(TSID_E_DEVICE, "hipGetSymbolAddress returned no address for the scratch array");
        g_scratch_ptr[device] = ptr;
    }
    return g_scratch_ptr[device];
}

// Bytes of the scratch the allocation-free loss needs: the reduction's
// partial sums and result (fp64), then per-item e^2 and the per-row norms of
// P and Q (fp32), each 256-byte aligned.
struct NoAllocLayout {
    size_t partial = 0, out = 0, e2 = 0, normP = 0, normQ = 0, total = 0;
};
NoAllocLayout noalloc_layout(int64_t n_items, int64_t m_t, int64_t n_t) {
    auto up = [](size_t b) { return (b + 255) & ~size_t(255); };
    NoAllocLayout L;
    L.partial = 0;
    L.out = up(L.partial + reduce_scratch_elems(1) * sizeof(double));
    L.e2 = up(L.out + sizeof(double));
    L.normP = up(L.e2 + (size_t)std::max<int64_t>(n_items, 1) * 4);
    L.normQ = up(L.normP + (size_t)std::max<int64_t>(m_t, 1) * 4);
    L.total = up(L.normQ + (size_t)std::max<int64_t>(n_t, 1) * 4);
    return L;
}

// tsid_loss with every buffer in the scratch array (the same kernels in the
// same order as loss(), so the result is the same bits).
void loss_noalloc(tsid_ctx *c, const float *P, const float *Q, float lambda, double *out) {
    if (!c->tpl) fail(TSID_E_STATE, "no template");
    Template &t = *c->tpl;
    if (!out) fail(TSID_E_INVAL, "out is NULL");
    if ((t.m_t && !P) || (t.n_t && !Q)) fail(TSID_E_INVAL, "NULL factor pointer");
    if (!(lambda >= 0.f) || !std::isfinite(lambda)) fail(TSID_E_INVAL, "lambda must be finite and >= 0");
    check_aligned(P, "P");
    check_aligned(Q, "Q");
    const Plan &pl = t.plan[0][TSID_FP32];
    if (!pl.ready) fail(TSID_E_STATE, "the template has no fp32 row plan");
    const NoAllocLayout L = noalloc_layout(pl.n_items, t.m_t, t.n_t);
    if (L.total > kNoAllocBytes)
        fail(TSID_E_NOMEM, "the allocation-free loss needs " + std::to_string(L.total) + " bytes of scratch (" +
                               "4 per work item, template row and column, plus 2 KiB); it has " +
                               std::to_string(kNoAllocBytes));
    char *base = static_cast<char *>(c->noalloc_scratch);
    if (!base) fail(TSID_E_STATE, "no scratch address for this device");
    double *partial = reinterpret_cast<double *>(base + L.partial);
    double *dout = reinterpret_cast<double *>(base + L.out);
    float *e2 = reinterpret_cast<float *>(base + L.e2);
    float *normP = reinterpret_cast<float *>(base + L.normP);
    float *normQ = reinterpret_cast<float *>(base + L.normQ);
    hipStream_t cs = c->comp;
    tsid_fit_opts o{0, lambda, 1.f, 1.f, 0, TSID_FP32, TSID_STEP_SUM};
    PassArgs a = pass_args(t, 0, o, c->err_dev);
    a.X = P;
    a.Y = Q;
    a.e2 = e2;
    a.norm = normP;
    a.epoch = 0;
    a.skip_after_nonfinite = 0;
    launch_item_pass(t.k, TSID_FP32, true, a, cs);
    launch_row_norms(t.k, Q, t.n_t, normQ, cs);
    launch_loss_reduce(e2, std::max<int64_t>(pl.n_items, 1), pl.n_items, normP, t.m_t, normQ, t.n_t, lambda, 1,
                       partial, dout, nullptr, -1, cs);
    TSID_HIP(hipMemcpyAsync(out, dout, 8, hipMemcpyDeviceToHost, cs));
    TSID_HIP(hipStreamSynchronize(cs));
}

// ------------------------------------------------------------- extension

void ext_sync_all(tsid_ctx *c) {
    TSID_HIP(hipStreamSynchronize(c->h2d));
    TSID_HIP(hipStreamSynchronize(c->comp));
    TSID_HIP(hipStreamSynchronize(c->d2h));
}

void ext_ensure(tsid_ctx *c, int64_t nnz, int32_t n_free, int32_t k) {
    ExtState &x = c->ext;
    Arena &A = c->arena;
    if (!x.slot[0].ev_h2d) {
        for (auto &s : x.slot) {
            TSID_HIP(hipEventCreateWithFlags(&s.ev_h2d, hipEventDisableTiming));
            TSID_HIP(hipEventCreateWithFlags(&s.ev_staged, hipEventDisableTiming));
            TSID_HIP(hipEventCreateWithFlags(&s.ev_done, hipEventDisableTiming));
            TSID_HIP(hipEventCreateWithFlags(&s.ev_flushed, hipEventDisableTiming));
        }
        x.err = A.alloc<int32_t>(ERR_SLOTS);
        TSID_HIP(hipMemsetAsync(x.err, 0, ERR_SLOTS * 4, c->comp));
        x.unsorted = A.alloc<uint32_t>(1);
    }
    if (nnz <= x.cap_nnz && n_free <= x.cap_free && k == x.k) return;
    ext_sync_all(c);  // buffers may be in use by earlier chunks
    const int64_t cn = std::max<int64_t>({nnz, x.cap_nnz + x.cap_nnz / 2, 1024});
    const int32_t cf = (int32_t)std::min<int64_t>(std::max<int64_t>({(int64_t)n_free, (int64_t)x.cap_free + x.cap_free / 2, 64}), INT32_MAX - 1);
    int32_t *err_keep = x.err;
    x.err = nullptr;
    free_ext_buffers(c);
    x.err = err_keep;
    for (auto &s : x.slot) {
        s.fid = A.alloc<int32_t>(cn);
        s.free_id = A.alloc<int32_t>(cn);
        s.r = A.alloc<float>(cn);
        s.X = A.alloc<float>((int64_t)cf * k);
    }
    x.keys = A.alloc<uint64_t>(cn);
    x.keys_alt = A.alloc<uint64_t>(cn);
    x.vals = A.alloc<uint32_t>(cn);
    x.vals_alt = A.alloc<uint32_t>(cn);
    x.sort_scratch = A.alloc<uint32_t>((int64_t)radix_scratch_elems(cn));
    x.stream = A.alloc<int2>(cn);
    x.ptr = A.alloc<int64_t>((int64_t)cf + 1);
    // items of at least 64 cells: at most one per row plus nnz / 64
    x.plan_cap = (int64_t)cf + cn / 64 + 1;
    x.plan_off = A.alloc<uint32_t>((int64_t)cf + 1);
    x.plan_nparts = A.alloc<uint32_t>(cf);
    x.plan_scan = A.alloc<uint32_t>((int64_t)scan_scratch_elems(cf));
    x.plan_items = A.alloc<int32_t>(x.plan_cap);
    x.plan_carry = A.alloc<float>(x.plan_cap * k);
    x.cap_nnz = cn;
    x.cap_free = cf;
    x.k = k;
}

// The Adam extension's request: options, basis and the optional C output.
struct AdamReq {
    const tsid_adam_opts *o;
    const float *basis;
    int64_t n_b;
    float *C_out;
};

// Per-slot Adam state for n_free x n_b coefficients (grown, never shrunk;
// growth waits for every chunk in flight, which may still read the old ones).
void adam_ensure(tsid_ctx *c, ExtSlot &s, int64_t n_free, int64_t n_b, int K) {
    const int64_t nc = std::max<int64_t>(n_free * n_b, 1), nq = std::max<int64_t>(n_free * adam_slices(n_b) * K, 1),
                  ng = std::max<int64_t>(n_free * K, 1);
    if (nc <= s.adam_cap && nq <= s.qpart_cap && ng <= s.gt_cap) return;
    ext_sync_all(c);
    Arena &A = c->arena;
    A.release(s.Cst);
    A.release(s.Mst);
    A.release(s.Vst);
    A.release(s.qpart);
    A.release(s.gt);
    s.adam_cap = s.qpart_cap = s.gt_cap = 0;
    s.Cst = A.alloc<float>(nc);
    s.Mst = A.alloc<float>(nc);
    s.Vst = A.alloc<float>(nc);
    s.qpart = A.alloc<float>(nq);
    s.gt = A.alloc<float>(ng);
    s.adam_cap = nc;
    s.qpart_cap = nq;
    s.gt_cap = ng;
}

// One chunk of the extension: staging, bucketing by free row, then the
// one-sided gradient steps of `o`, or (ridge != null) the exact solve with
// lambda = *ridge, or (adam != null) Adam on the coefficients in a basis.
// Adds a finished chunk's copy and compute durations to the timing totals.
void ext_take_timing(tsid_ctx *c, ExtSlot &s) {
    if (!s.tm_pending) return;
    float h = 0.f, k = 0.f;
    TSID_HIP(hipEventElapsedTime(&h, s.tm[0], s.tm[1]));
    TSID_HIP(hipEventElapsedTime(&k, s.tm[2], s.tm[3]));
    c->tm.ext_h2d_ms += h;
    c->tm.ext_compute_ms += k;
    c->tm.ext_chunks += 1;
    s.tm_pending = false;
}

void extend_chunk(tsid_ctx *c, int side, const int32_t *fixed_id, const int32_t *free_local,
                  const float *r, int64_t nnz, int32_t n_free, const float *F_fixed, int64_t n_fixed,
                  float *F_free, const tsid_fit_opts *o, const float *ridge, const AdamReq *adam = nullptr) {
    if (!c->tpl) fail(TSID_E_STATE, "no template: the rank k is set by tsid_build_template");
    if (adam) {
        const tsid_adam_opts *ao = adam->o;
        if (!ao) fail(TSID_E_INVAL, "opts is NULL");
        if (ao->steps < 0) fail(TSID_E_INVAL, "steps < 0");
        if (!(ao->lambda >= 0.f) || !std::isfinite(ao->lambda)) fail(TSID_E_INVAL, "lambda must be finite and >= 0");
        if (!std::isfinite(ao->lr)) fail(TSID_E_INVAL, "lr must be finite");
        if (!(ao->beta1 >= 0.f && ao->beta1 < 1.f) || !(ao->beta2 >= 0.f && ao->beta2 < 1.f))
            fail(TSID_E_INVAL, "beta1 and beta2 must lie in [0, 1)");
        if (!(ao->eps >= 0.f) || !std::isfinite(ao->eps)) fail(TSID_E_INVAL, "eps must be finite and >= 0");
        if (!adam_supported(c->tpl->k)) fail(TSID_E_INVAL, "the Adam extension supports k in {8, 16, 32, 64, 128}");
        if (adam->n_b < 1 || adam->n_b >= (int64_t(1) << 31)) fail(TSID_E_INVAL, "n_basis out of range");
        if (!adam->basis) fail(TSID_E_INVAL, "basis is NULL");
        check_aligned(adam->basis, "basis");
    } else if (ridge) {
        if (!(*ridge >= 0.f) || !std::isfinite(*ridge)) fail(TSID_E_INVAL, "lambda must be finite and >= 0");
        if (!ridge_supported(c->tpl->k)) fail(TSID_E_INVAL, "the exact extension solve supports k in {8, 16, 32, 64, 128}");
    } else {
        check_opts(o);
        if (o->clip == 2) fail(TSID_E_INVAL, "per-entry clipping (clip 2) is a template-fit option");
        if (o->step == TSID_STEP_COL_DEGREE)
            fail(TSID_E_INVAL, "the column-only degree step is a template-fit option");
    }
    if (side != 0 && side != 1) fail(TSID_E_INVAL, "side must be 0 or 1");
    if (nnz < 0 || nnz > kMaxEntries) fail(TSID_E_INVAL, "nnz out of range");
    if (n_free < 0 || n_fixed < 0 || n_fixed >= (int64_t(1) << 31)) fail(TSID_E_INVAL, "bad sizes");
    if (nnz > 0 && (!fixed_id || !free_local || !r)) fail(TSID_E_INVAL, "NULL chunk arrays");
    if (nnz > 0 && (!F_fixed || n_fixed == 0)) fail(TSID_E_INVAL, "no fixed factors");
    if (n_free > 0 && !F_free) fail(TSID_E_INVAL, "F_free is NULL");
    if (F_fixed) check_aligned(F_fixed, "F_fixed");
    const int K = c->tpl->k;
    ext_ensure(c, nnz, n_free, K);
    ExtState &x = c->ext;
    const int si = x.next;
    x.next ^= 1;
    ExtSlot &s = x.slot[si];
    hipStream_t cs = c->comp;
    const bool tmo = c->timing > 0;
    if (tmo) {
        if (s.tm_pending) {  // the slot's previous chunk: finished before its events are reused
            TSID_HIP(hipEventSynchronize(s.tm[3]));
            ext_take_timing(c, s);
        }
        for (auto &e : s.tm)
            if (!e) TSID_HIP(hipEventCreate(&e));
    }
    // stage the chunk (copy stream), after the slot's previous chunk consumed it
    TSID_HIP(hipStreamWaitEvent(c->h2d, s.ev_staged, 0));
    if (tmo) TSID_HIP(hipEventRecord(s.tm[0], c->h2d));
    if (nnz) {
        TSID_HIP(hipMemcpyAsync(s.fid, fixed_id, (size_t)nnz * 4, hipMemcpyHostToDevice, c->h2d));
        TSID_HIP(hipMemcpyAsync(s.free_id, free_local, (size_t)nnz * 4, hipMemcpyHostToDevice, c->h2d));
        TSID_HIP(hipMemcpyAsync(s.r, r, (size_t)nnz * 4, hipMemcpyHostToDevice, c->h2d));
    }
    TSID_HIP(hipEventRecord(s.ev_h2d, c->h2d));
    if (tmo) TSID_HIP(hipEventRecord(s.tm[1], c->h2d));
    TSID_HIP(hipStreamWaitEvent(cs, s.ev_h2d, 0));
    if (tmo) TSID_HIP(hipEventRecord(s.tm[2], cs));
    // bucket the chunk by free row: key = free << bits_fixed | fixed (stable sort)
    const int bits_fixed = bits_for(std::max<int64_t>(n_fixed, 1));
    const int bits_free = bits_for(std::max<int32_t>(n_free, 1));
    chunk_keys(s.fid, s.free_id, s.r, nnz, n_fixed, n_free, bits_fixed, x.keys, x.vals, x.err, cs);
    TSID_HIP(hipEventRecord(s.ev_staged, cs));
    // a chunk already grouped by free row (fixed ids ascending within a row,
    // as a line-by-line generator emits them) skips the sort's passes
    keys_unsorted(x.keys, nnz, x.unsorted, cs);
    const bool alt = radix_sort(x.keys, x.vals, x.keys_alt, x.vals_alt, nnz, bits_fixed + bits_free,
                                x.sort_scratch, cs, x.unsorted);
    const uint64_t *sk = alt ? x.keys_alt : x.keys;
    const uint32_t *sv = alt ? x.vals_alt : x.vals;
    keys_to_stream(sk, sv, nnz, bits_fixed, x.stream, x.err, cs);
    ptr_from_keys(sk, nnz, n_free, bits_fixed, x.ptr, cs);
    // the slot's result buffer is free once its previous results were flushed
    TSID_HIP(hipStreamWaitEvent(cs, s.ev_flushed, 0));
    if (adam) {
        adam_ensure(c, s, n_free, adam->n_b, K);
        const int64_t nc = (int64_t)n_free * adam->n_b, nq = (int64_t)n_free * adam_slices(adam->n_b) * K;
        if (nc) {
            TSID_HIP(hipMemsetAsync(s.Cst, 0, (size_t)nc * 4, cs));
            TSID_HIP(hipMemsetAsync(s.Mst, 0, (size_t)nc * 4, cs));
            TSID_HIP(hipMemsetAsync(s.Vst, 0, (size_t)nc * 4, cs));
            TSID_HIP(hipMemsetAsync(s.qpart, 0, (size_t)nq * 4, cs));
        }
        AdamArgs a{};
        a.stream = x.stream;
        a.ptr = x.ptr;
        a.n_free = n_free;
        a.F = F_fixed;
        a.B = adam->basis;
        a.n_b = adam->n_b;
        a.n_slices = adam_slices(adam->n_b);
        a.C = s.Cst;
        a.M = s.Mst;
        a.V = s.Vst;
        a.qpart = s.qpart;
        a.gt = s.gt;
        a.X = s.X;
        a.lambda = adam->o->lambda;
        a.lr = adam->o->lr;
        a.beta1 = adam->o->beta1;
        a.beta2 = adam->o->beta2;
        a.eps = adam->o->eps;
        a.err = x.err;
        a.skip_after_nonfinite = 1;
        // the gradient of every step runs on the item pass: its work plan
        // (items of at most E cells of a free line) built on the device
        const int32_t E = choose_E(nnz);
        plan_items(x.ptr, n_free, E, x.plan_off, x.plan_items, x.plan_nparts, x.plan_scan, cs);
        a.item_off = x.plan_off;
        a.items = x.plan_items;
        a.n_items_ub = (int64_t)n_free + nnz / E + 1;
        a.E = E;
        a.carry = x.plan_carry;
        a.n_fixed = n_fixed;
        launch_adam(K, a, adam->o->steps, cs);
    } else if (ridge) {
        RidgeArgs a{};
        a.stream = x.stream;
        a.ptr = x.ptr;
        a.rows = n_free;
        a.F = F_fixed;
        a.lambda = *ridge;
        a.X = s.X;
        a.err = x.err;
        launch_ridge_rows(K, a, cs);  // one wave per free row
    } else {
        PassArgs a{};
        a.stream = x.stream;
        a.ptr = x.ptr;
        a.rows = n_free;
        a.Y = F_fixed;
        a.y_rows = n_fixed;
        a.Xn = s.X;
        a.lam = o->lambda;
        a.lr = o->lr;
        a.xi = o->clip_xi;
        a.clip = o->clip;
        a.degree = o->step == TSID_STEP_DEGREE;
        a.err = x.err;
        // rows long enough for the Gram form go to k_extend_gram, the others
        // take every step in one launch of the per-cell kernel (one wave per
        // free row in both)
        const int64_t gmin = extend_gram_min(K, o->epochs, o->clip, n_fixed);
        a.skip_from = gmin;
        launch_extend_steps(K, a, o->epochs, cs);
        if (gmin > 0) {
            RidgeArgs g{};
            g.stream = x.stream;
            g.ptr = x.ptr;
            g.rows = n_free;
            g.F = F_fixed;
            g.lambda = o->lambda;
            g.X = s.X;
            g.err = x.err;
            g.gram_min = gmin;
            g.steps = o->epochs;
            g.clip = o->clip;
            g.degree = a.degree;
            g.lr = o->lr;
            g.xi = o->clip_xi;
            launch_extend_gram(K, g, cs);
        }
    }
    if (tmo) {
        TSID_HIP(hipEventRecord(s.tm[3], cs));
        s.tm_pending = true;
    }
    TSID_HIP(hipEventRecord(s.ev_done, cs));
    // flush the results on the third stream
    TSID_HIP(hipStreamWaitEvent(c->d2h, s.ev_done, 0));
    if (n_free)
        // host or device memory: the runtime takes the direction from the address
        TSID_HIP(hipMemcpyAsync(F_free, s.X, (size_t)n_free * K * 4, hipMemcpyDefault, c->d2h));
    if (adam && adam->C_out && n_free)
        TSID_HIP(hipMemcpyAsync(adam->C_out, s.Cst, (size_t)n_free * adam->n_b * 4, hipMemcpyDefault, c->d2h));
    TSID_HIP(hipEventRecord(s.ev_flushed, c->d2h));
    x.pending = true;
    // The previous chunk (the other slot) was queued before this one; once
    // its host-to-device copy has finished, its host input arrays are free
    // for the caller to refill, so two pinned host buffers can feed the
    // stream while this chunk's copy and the previous chunk's compute run.
    TSID_HIP(hipEventSynchronize(x.slot[si ^ 1].ev_h2d));
    (void)side;
}

void sync(tsid_ctx *c) {
    ext_sync_all(c);
    for (auto &s : c->ext.slot) ext_take_timing(c, s);
    ExtState &x = c->ext;
    if (!x.err) return;
    int32_t e[ERR_SLOTS];
    TSID_HIP(hipMemcpy(e, x.err, sizeof(e), hipMemcpyDeviceToHost));
    TSID_HIP(hipMemset(x.err, 0, sizeof(e)));
    x.pending = false;
    raise_device_errors(e, "extend");
    if (e[ERR_NONFINITE]) fail(TSID_E_NONFINITE, "extend: non-finite update");
}

void export_index(const tsid_ctx *c, int which, void *dst, size_t bytes) {
    if (!c->tpl) fail(TSID_E_STATE, "no template");
    if (!dst && bytes) fail(TSID_E_INVAL, "host_dst is NULL");
    const Template &t = *c->tpl;
    auto need = [&](size_t want) {
        if (bytes != want) fail(TSID_E_INVAL, "bytes must be " + std::to_string(want));
    };
    auto copy = [&](const void *src, size_t n) {
        if (n) TSID_HIP(hipMemcpy(dst, src, n, hipMemcpyDeviceToHost));
    };
    auto split = [&](const int2 *stream, int part) {
        need((size_t)t.nnz * 4);
        std::vector<int2> h((size_t)t.nnz);
        copy(nullptr, 0);
        if (t.nnz) TSID_HIP(hipMemcpy(h.data(), stream, (size_t)t.nnz * 8, hipMemcpyDeviceToHost));
        int32_t *o = static_cast<int32_t *>(dst);
        for (int64_t j = 0; j < t.nnz; ++j) o[j] = part ? h[j].y : h[j].x;
    };
    auto degrees = [&](const int64_t *ptr, int32_t rows) {
        need((size_t)rows * 4);
        std::vector<int64_t> h((size_t)rows + 1);
        TSID_HIP(hipMemcpy(h.data(), ptr, (size_t)(rows + 1) * 8, hipMemcpyDeviceToHost));
        int32_t *o = static_cast<int32_t *>(dst);
        for (int32_t x = 0; x < rows; ++x) o[x] = (int32_t)(h[x + 1] - h[x]);
    };
    switch (which) {
        case TSID_IDX_ROW_MAP: need((size_t)t.m * 4); copy(t.row_map, (size_t)t.m * 4); break;
        case TSID_IDX_COL_MAP: need((size_t)t.n * 4); copy(t.col_map, (size_t)t.n * 4); break;
        case TSID_IDX_ROW_PTR: need((size_t)(t.m_t + 1) * 8); copy(t.row_ptr, (size_t)(t.m_t + 1) * 8); break;
        case TSID_IDX_COL_PTR: need((size_t)(t.n_t + 1) * 8); copy(t.col_ptr, (size_t)(t.n_t + 1) * 8); break;
        case TSID_IDX_CSR_COL: split(t.stream_r, 0); break;
        case TSID_IDX_CSR_VAL: split(t.stream_r, 1); break;
        case TSID_IDX_CSC_ROW: split(t.stream_c, 0); break;
        case TSID_IDX_CSC_VAL: split(t.stream_c, 1); break;
        case TSID_IDX_DEG_R: degrees(t.row_ptr, t.m_t); break;
        case TSID_IDX_DEG_C: degrees(t.col_ptr, t.n_t); break;
        case TSID_IDX_BATCH_PTR_R:
        case TSID_IDX_BATCH_PTR_C: {
            const int sd = which == TSID_IDX_BATCH_PTR_C;
            if (!t.mb.ready) fail(TSID_E_STATE, "no mini-batch fit has run on this template");
            need(t.mb.hptr[sd].size() * 8);
            std::memcpy(dst, t.mb.hptr[sd].data(), bytes);
            break;
        }
        default: fail(TSID_E_INVAL, "unknown index structure");
    }
}

}  // namespace

// ================================================================ C ABI

extern "C" {

tsid_status tsid_create(int device, void *hip_stream, size_t max_device_bytes, tsid_ctx **out) {
    if (!out) return TSID_E_INVAL;
    *out = nullptr;
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device < 0 || device >= count) {
        (void)hipGetLastError();
        return TSID_E_DEVICE;
    }
    tsid_ctx *c = new tsid_ctx;
    c->device = device;
    c->arena.cap = max_device_bytes;
    tsid_status st = guarded(c, [&]() {
        if (hip_stream) {
            c->comp = static_cast<hipStream_t>(hip_stream);
        } else {
            TSID_HIP(hipStreamCreateWithFlags(&c->comp, hipStreamDefault));
            c->own_comp = true;
        }
        TSID_HIP(hipStreamCreateWithFlags(&c->h2d, hipStreamDefault));
        TSID_HIP(hipStreamCreateWithFlags(&c->d2h, hipStreamDefault));
        c->err_dev = c->arena.alloc<int32_t>(ERR_SLOTS);
        TSID_HIP(hipHostMalloc((void **)&c->err_host, ERR_SLOTS * sizeof(int32_t), hipHostMallocDefault));
        TSID_HIP(hipMemset(c->err_dev, 0, ERR_SLOTS * sizeof(int32_t)));
        c->noalloc_scratch = noalloc_scratch_on(device);
    });
    if (st != TSID_OK) {
        tsid_destroy(c);
        return st;
    }
    *out = c;
    return TSID_OK;
}

void tsid_destroy(tsid_ctx *c) {
    if (!c) return;
    (void)hipSetDevice(c->device);
    if (c->h2d) (void)hipStreamSynchronize(c->h2d);
    if (c->comp) (void)hipStreamSynchronize(c->comp);
    if (c->d2h) (void)hipStreamSynchronize(c->d2h);
    free_template(c, c->tpl);
    free_fit(c);
    free_ext_buffers(c);
    c->arena.release(c->ext.err);
    c->arena.release(c->ext.unsorted);
    for (auto &s : c->ext.slot) {
        if (s.ev_h2d) (void)hipEventDestroy(s.ev_h2d);
        if (s.ev_staged) (void)hipEventDestroy(s.ev_staged);
        if (s.ev_done) (void)hipEventDestroy(s.ev_done);
        if (s.ev_flushed) (void)hipEventDestroy(s.ev_flushed);
        for (auto &e : s.tm)
            if (e) (void)hipEventDestroy(e);
    }
    for (hipEvent_t e : c->events) (void)hipEventDestroy(e);
    c->arena.release(c->err_dev);
    if (c->err_host) (void)hipHostFree(c->err_host);
    if (c->h2d) (void)hipStreamDestroy(c->h2d);
    if (c->d2h) (void)hipStreamDestroy(c->d2h);
    if (c->own_comp && c->comp) (void)hipStreamDestroy(c->comp);
    delete c;
}

const char *tsid_last_error(const tsid_ctx *c) { return c ? c->err.c_str() : "NULL context"; }

tsid_status tsid_build_template(tsid_ctx *c, int64_t m, int64_t n, const int32_t *u, const int32_t *i,
                                const float *r, int64_t nnz, const int32_t *I, int32_t m_t,
                                const int32_t *J, int32_t n_t, int32_t k, int64_t stage_entries) {
    return guarded(c, [&]() { build(c, m, n, u, i, r, nnz, I, m_t, J, n_t, k, stage_entries); });
}

tsid_status tsid_template_info(const tsid_ctx *c, int32_t *m_t, int32_t *n_t, int64_t *nnz, int32_t *k) {
    if (!c) return TSID_E_INVAL;
    if (!c->tpl) return TSID_E_STATE;
    if (m_t) *m_t = c->tpl->m_t;
    if (n_t) *n_t = c->tpl->n_t;
    if (nnz) *nnz = c->tpl->nnz;
    if (k) *k = c->tpl->k;
    return TSID_OK;
}

tsid_status tsid_fit_template(tsid_ctx *c, float *P, float *Q, const tsid_fit_opts *opts,
                              double *loss_hist) {
    return guarded(c, [&]() { fit(c, P, Q, opts, loss_hist); });
}

tsid_status tsid_set_pass_kernel(tsid_ctx *c, int mode) {
    return guarded(c, [&]() {
        if (mode != TSID_PASS_AUTO && mode != TSID_PASS_ITEM && mode != TSID_PASS_SLAB)
            fail(TSID_E_INVAL, "unknown pass kernel mode");
        c->pass_kernel = mode;
    });
}

tsid_status tsid_fit_pass_kernels(const tsid_ctx *c, int32_t *p_pass, int32_t *q_pass) {
    if (!c) return TSID_E_INVAL;
    if (p_pass) *p_pass = c->used_kernel[0];
    if (q_pass) *q_pass = c->used_kernel[1];
    return TSID_OK;
}

tsid_status tsid_set_dense_tiles(tsid_ctx *c, float fill) {
    if (!c || !(fill <= 1.f)) return TSID_E_INVAL;  // NaN fails the comparison
    c->dense_fill = fill < 0.f ? -1.f : fill;
    return TSID_OK;
}

tsid_status tsid_set_similarity(tsid_ctx *c, const int32_t *row, const int32_t *col, const float *val,
                                int64_t nnz, float beta) {
    return guarded(c, [&]() { set_similarity(c, row, col, val, nnz, beta); });
}

tsid_status tsid_set_row_blocks(tsid_ctx *c, int32_t n_blocks) {
    if (!c || n_blocks < 0 || n_blocks > TSID_MAX_ROW_BLOCKS) return TSID_E_INVAL;
    c->row_blocks = n_blocks;
    return TSID_OK;
}

tsid_status tsid_fit_row_blocks(const tsid_ctx *c, int32_t *n_blocks) {
    if (!c || !n_blocks) return TSID_E_INVAL;
    *n_blocks = c->used_blocks;
    return TSID_OK;
}

tsid_status tsid_set_minibatch(tsid_ctx *c, int32_t n_batches, uint64_t seed) {
    if (!c || n_batches < 0 || n_batches > TSID_MAX_BATCHES) return TSID_E_INVAL;
    c->mb_batches = n_batches;
    c->mb_seed = seed;
    return TSID_OK;
}

tsid_status tsid_fit_dense_info(const tsid_ctx *c, tsid_dense_info *out) {
    if (!c || !out) return TSID_E_INVAL;
    *out = c->dense_used;
    return TSID_OK;
}

tsid_status tsid_set_timing(tsid_ctx *c, int every) {
    if (!c || every < 0) return TSID_E_INVAL;
    return guarded(c, [&] {
        if (every > 0) grow_events(c, kEventPool);
        c->timing = every;
        c->tm = tsid_timing{};
    });
}

tsid_status tsid_get_timing(const tsid_ctx *c, tsid_timing *out) {
    if (!c || !out) return TSID_E_INVAL;
    *out = c->tm;
    return TSID_OK;
}

tsid_status tsid_fit_epochs_done(const tsid_ctx *c, int32_t *epochs) {
    if (!c || !epochs) return TSID_E_INVAL;
    *epochs = c->epochs_done;
    return TSID_OK;
}

tsid_status tsid_loss_noalloc(tsid_ctx *c, const float *P, const float *Q, float lambda, double *out) {
    return guarded(c, [&]() { loss_noalloc(c, P, Q, lambda, out); });
}

tsid_status tsid_loss(tsid_ctx *c, const float *P, const float *Q, float lambda, double *out) {
    return guarded(c, [&]() { loss(c, P, Q, lambda, out); });
}

tsid_status tsid_extend_chunk(tsid_ctx *c, int side, const int32_t *fixed_id, const int32_t *free_local,
                              const float *r, int64_t nnz, int32_t n_free, const float *F_fixed,
                              int64_t n_fixed, float *F_free, const tsid_fit_opts *opts) {
    return guarded(c, [&]() {
        extend_chunk(c, side, fixed_id, free_local, r, nnz, n_free, F_fixed, n_fixed, F_free, opts, nullptr);
    });
}

tsid_status tsid_extend_chunk_adam(tsid_ctx *c, int side, const int32_t *fixed_id, const int32_t *free_local,
                                   const float *r, int64_t nnz, int32_t n_free, const float *F_fixed,
                                   int64_t n_fixed, const float *basis, int64_t n_basis, float *F_free,
                                   float *C_out, const tsid_adam_opts *opts) {
    return guarded(c, [&]() {
        const AdamReq req{opts, basis, n_basis, C_out};
        extend_chunk(c, side, fixed_id, free_local, r, nnz, n_free, F_fixed, n_fixed, F_free, nullptr, nullptr,
                     &req);
    });
}

tsid_status tsid_extend_chunk_ridge(tsid_ctx *c, int side, const int32_t *fixed_id, const int32_t *free_local,
                                    const float *r, int64_t nnz, int32_t n_free, const float *F_fixed,
                                    int64_t n_fixed, float *F_free, float lambda) {
    return guarded(c, [&]() {
        extend_chunk(c, side, fixed_id, free_local, r, nnz, n_free, F_fixed, n_fixed, F_free, nullptr, &lambda);
    });
}

tsid_status tsid_sync(tsid_ctx *c) {
    return guarded(c, [&]() { sync(c); });
}

tsid_status tsid_export_index(const tsid_ctx *c, int which, void *host_dst, size_t bytes) {
    tsid_ctx *mc = const_cast<tsid_ctx *>(c);
    return guarded(mc, [&]() { export_index(c, which, host_dst, bytes); });
}

int32_t tsid_chunk_plan(const int64_t *counts, int64_t n_free, int32_t n_chunks, int64_t max_entries,
                        int64_t *bounds, int32_t max_bounds) {
    if (n_free < 0 || (n_free > 0 && !counts) || !bounds || max_bounds < 1 || n_chunks < 0) return -1;
    if (n_chunks == 0 && max_entries <= 0) return -1;
    for (int64_t f = 0; f < n_free; ++f)
        if (counts[f] < 0) return -1;
    if (n_chunks > 0) {
        if (max_bounds < n_chunks + 1) return -1;
        // prefix of cells before each row; run j starts where the prefix first
        // reaches ceil(j * total / n_chunks)
        __int128 total = 0;
        for (int64_t f = 0; f < n_free; ++f) total += counts[f];
        int64_t f = 0;
        __int128 before = 0;
        for (int32_t j = 0; j < n_chunks; ++j) {
            const __int128 target = (total * j + n_chunks - 1) / n_chunks;
            while (f < n_free && before < target) before += counts[f++];
            bounds[j] = f;
        }
        bounds[n_chunks] = n_free;
        return n_chunks;
    }
    int32_t runs = 0;
    bounds[0] = 0;
    int64_t f = 0;
    while (f < n_free) {
        int64_t cells = counts[f++];
        while (f < n_free && cells + counts[f] <= max_entries) cells += counts[f++];
        if (runs + 2 > max_bounds) return -1;
        bounds[++runs] = f;
    }
    return runs;
}

}  // extern "C"
