#!/usr/bin/env python3
"""Throughput of the TSID template fit (Stage I, Section 5.1) on one MI355X.

A step is one full-gradient epoch of the template fit: the P pass over the
row buckets, the Q pass over the column buckets, the fixups of buckets longer
than one wave (when the template has any) and the epoch's share of the
loss-history reduction (the fit runs with its loss history on, as it does when
it is run until convergence; the loss of the final iterate is computed inside
the timed region too).
The metric is observed template cells per second per epoch
(|Omega*_train| / epoch time).  Inputs are resident in HBM before the timed
region starts; the template build (host stream, filter, bucketing) is timed
separately and reported as build_s.

Default workload: the Billion-scale configuration's template, the largest
workload that fits one GPU -- the 1,000,000 x 100,000 most-popular template of
a 10 M x 1 M Zipf(1.0) matrix with 1e9 observed cells (about 4.2e8 training
cells in the template), k = 128, bf16 factors with fp32 accumulation and the
asymmetric clip, degree step.  --config scientific runs the 16,384 x 16,384
uniform template of the 200,000 x 200,000 rank-32 matrix (k = 32, fp32);
--config rating the Netflix-shaped template (65,536 x 8,192, k = 64, bf16);
mid / tiny are small.

Roofline: every kernel kind of an epoch (the P and Q passes or their one
paired launch, the dense-tile launches) is priced with the algorithmic work
of the cells it covers: per observed cell and epoch, 12 bytes (each
(u, i, r) read once) and 6k flops (one dot product, two axpys), a launch of
one pass taking half of both, plus each owner row it updates read and
written once (fp32 master; in bf16 mode its bf16 copy written too).  The
fractions of the MI355X peaks (HBM 8 TB/s, fp32 vector 157.3 TFLOP/s, bf16
matrix cores 2.5 PFLOP/s for the dense-tile kernels) are reported for each;
the roofline object is the kernel with the most time per epoch, bound by the
unit with the highest fraction.  Durations come from HIP events attached to
the dispatches on the library's compute stream during the timed region
(every --time-every-th epoch: a timed dispatch costs a few microseconds of
wall time, which would otherwise slow the throughput being measured).

CPU baseline: the fp64 oracle built with OpenMP on all host cores (the
line-parallel fit, the same bits as the serial oracle) on a bounded sample of
the same template cells, for as many epochs as fit in about --cpu-seconds.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)



def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="billion", choices=["scientific", "rating", "billion", "mid", "tiny"])
    ap.add_argument("--pass-kernel", default="auto", choices=["auto", "item", "slab"],
                    help="kernel of the P and Q passes (tsid_set_pass_kernel); auto picks the "
                         "slab pass for evenly spread fp32 templates")
    ap.add_argument("--dense-fill", type=float, default=-1.0,
                    help="dense head tiles of bf16 fits (tsid_set_dense_tiles): < 0 automatic, "
                         "0 off, in (0, 1] forced with that tile fill")
    ap.add_argument("--clip-per-entry", action="store_true",
                    help="the clip in the per-entry order (fit option clip = 2; item pass, no tiles)")
    ap.add_argument("--similarity", type=float, default=0.0,
                    help="beta of the multi-view term over a synthetic similarity graph of the template's "
                         "columns (16 random links per column, made mutual); item pass")
    ap.add_argument("--lr", type=float, default=None, help="step size instead of the workload's")
    ap.add_argument("--row-blocks", type=int, default=0,
                    help="row blocks of the item Q pass (tsid_set_row_blocks): 0 automatic, 1 off, n forced")
    ap.add_argument("--minibatch", type=int, default=0,
                    help="mini-batch epochs with this many batches (tsid_set_minibatch; 0: full-gradient "
                         "epochs); the batch steps run the item pass, the epochs' loss passes may take the "
                         "dense tiles of bf16 fits")
    ap.add_argument("--minibatch-seed", type=int, default=1)
    ap.add_argument("--time-every", type=int, default=10,
                    help="attach HIP timing events to the kernels of every n-th timed epoch (each "
                         "timed dispatch costs a few microseconds of wall time)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extend", action="store_true",
                    help="after the timed fit, time the end-to-end extension (row phase, then "
                         "column phase, streamed in chunks from pinned host memory) and print a "
                         "second JSON line with the PCIe fraction and the copy/compute overlap; on "
                         "Scientific and Billion-scale the cells outside the template come from the "
                         "streaming generator, filled into pinned memory before the timed run")
    ap.add_argument("--extend-steps", type=int, default=20)
    ap.add_argument("--extend-chunk", type=int, default=0,
                    help="cells per chunk of the streamed extension (0: 2^28 on Scientific, 2^26 on "
                         "Billion-scale)")
    ap.add_argument("--extend-solver", default="steps", choices=["steps", "ridge", "adam"],
                    help="extension solver: one-sided gradient steps (tsid_extend_chunk), the "
                         "exact ridge solve per free row (tsid_extend_chunk_ridge, fp64 Gram on the "
                         "matrix cores + Cholesky), or the column phase as Eq. 6 states it (Adam "
                         "on each free column's coefficients over the template columns' factors, "
                         "--extend-steps steps, lr 0.01; rows by the exact solve); all with the "
                         "fit's lambda")
    ap.add_argument("--copy-probe", action="store_true",
                    help="time a plain device copy of 1 GiB instead (HBM probe and the "
                         "reference kernel for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    return ap.parse_args()


def copy_probe(reps=20, nbytes=1 << 30):
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    moved = 2 * nbytes * reps
    print(json.dumps({"probe": "device copy", "bytes_read_per_launch": nbytes,
                      "bytes_written_per_launch": nbytes, "launches": reps + 3,
                      "GBps_read_plus_write": moved / el / 1e9}), flush=True)
    return 0


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Peaks of one MI355X (published figures): HBM3E bandwidth, the fp32 vector
# rate (the item and slab passes' arithmetic, fp32 or bf16 dot2 with fp32
# accumulation) and the dense bf16 matrix-core rate (the dense-tile kernels).
PEAK = {"hbm": (8000.0, "GB/s"), "alu": (157.3, "TFLOP/s"), "mfma": (2500.0, "TFLOP/s")}


def algorithmic(cells, owners, k, prec, sides=1, factor_rows=True):
    """Algorithmic bytes and flops of one launch covering `sides` passes
    (1: the P or the Q pass, 2: both) over `cells` observed cells: per cell
    and epoch each (u, i, r) is read once (12 B) and the work is one dot
    product and two axpys (6k flops), so a launch of one pass owns half of
    that; each owner row it updates is read once and written once (fp32
    master; in bf16 mode also its bf16 copy written).  `owners` is the owner
    row count of those passes together."""
    by = 6 * sides * cells
    if factor_rows:
        by += owners * (4 * k + 4 * k + (2 * k if prec == "bf16" else 0))
    return by, 3 * k * sides * cells


def roofline_of(ms, by, fl, units):
    """Fractions of the peaks for a launch of `ms` milliseconds moving `by`
    algorithmic bytes and doing `fl` algorithmic flops; the bound is the unit
    with the highest fraction among `units`."""
    s = ms / 1e3
    got = {"hbm": by / s / 1e9, "alu": fl / s / 1e12, "mfma": fl / s / 1e12}
    fr = {u: got[u] / PEAK[u][0] for u in units}
    bound = max(fr, key=fr.get)
    return bound, got[bound], fr


def traffic_from_profiles(kernel_src_sha, which):
    """Measured HBM bytes per launch, from the committed counter summary, if it
    was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    ent = d.get(which)
    if not ent or ent.get("kernel_source_sha256") != kernel_src_sha:
        return None
    return ent.get("hbm_bytes_per_launch")


def cpu_baseline(p, seconds, batches=0, seed=0):
    """The oracle timed on the host's cores: the line-parallel fp64 fit
    (or_fit_lines, OpenMP over all cores; the same bits as the serial fit) on
    a bounded sample of the template cells, with every template factor row,
    for as many epochs as fit in about `seconds`.  Mini-batch epochs have no
    parallel oracle and run the serial one."""
    import numpy as np

    import oracle
    st, rm, cm = oracle.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle.filter_template(p.u, p.i, p.r, rm, cm)
    S = int(min(a.size, 20_000_000 if not batches else 2_000_000))
    a, b, v = a[:S], b[:S], v[:S]
    cores = 1
    if batches:
        run = lambda ep: oracle.fit_minibatch(a, b, v, p.P0, p.Q0, ep, p.lam, p.lr, p.step, p.clip, p.xi,
                                              bf16=p.prec == "bf16", n_batches=batches, seed=seed)
        how = f"mini-batch epochs ({batches} batches), serial fp64 C"
    else:
        cores = oracle.threads(True)
        run = lambda ep: oracle.fit_lines(a, b, v, p.P0, p.Q0, ep, p.lam, p.lr, p.step, p.clip, p.xi,
                                          bf16=p.prec == "bf16", omp=True)
        how = (f"full-gradient epochs, fp64 C built with OpenMP ({cores} threads: rows, then columns, "
               f"split across threads; the same bits as the serial oracle)")
    t0 = time.perf_counter()
    run(1)
    one = time.perf_counter() - t0
    epochs = max(1, int(seconds / max(one, 1e-3)))
    t0 = time.perf_counter()
    run(epochs)
    el = time.perf_counter() - t0
    # epochs + 1 loss evaluations: the final one costs about a third of an epoch
    return {"value": S * epochs / el, "unit": "entries/s", "cores": cores, "kind": "oracle",
            "sample": f"first {S} template cells (input order, i.e. a uniform random sample) of "
                      f"the same workload, all {p.I.size} x {p.J.size} template factor rows, "
                      f"{epochs} {how}",
            "seconds": el, "nproc": os.cpu_count(), "cpu": _cpu_model()}


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def h2d_probe(nbytes, reps=5):
    """Pinned host-to-device copy rate (bytes/s) for a buffer of nbytes."""
    import torch
    src = torch.empty(nbytes // 4, dtype=torch.float32).pin_memory()
    dst = torch.empty_like(src, device="cuda")
    dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src, non_blocking=True)
    torch.cuda.synchronize()
    return nbytes * reps / (time.perf_counter() - t0)


def extension_line(args, p, T, P, Q):
    """End-to-end extension from the fitted template factors (Section 5.2)."""
    import torch

    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.extension import Extension, StreamedExtension
    streamed = p.extra.get("omega_scope") == "template block only"
    col_opts = None
    if args.extend_solver == "ridge":
        opts = float(p.lam)  # exact solve per free row
        how = f"exact ridge solve per free row (lambda {p.lam}, fp64 Gram + Cholesky)"
    elif args.extend_solver == "adam":
        if streamed:
            raise SystemExit("--extend-solver adam runs on the workloads whose whole matrix is drawn")
        opts = float(p.lam)
        col_opts = tsid.make_adam_opts(args.extend_steps, p.lam, 0.01)
        how = (f"rows by the exact ridge solve; columns by {args.extend_steps} Adam steps on their "
               f"coefficients over the {p.J.size} template columns' factors (Eq. 6; lr 0.01, "
               f"lambda {p.lam})")
    else:
        # one-sided steps from zero: lr 0.05 keeps a free row with a single cell stable
        opts = tsid.make_opts(epochs=args.extend_steps, lam=p.lam, lr=0.05, clip=p.clip, xi=p.xi,
                              step="degree")
        how = f"{args.extend_steps} one-sided steps per chunk, degree step"
    t0 = time.perf_counter()
    if streamed:
        import tsid_synth
        omega = tsid_synth.omega_outside_template(p)
        rows, cols = omega.row_phase(), omega.col_phase()
        max_entries = args.extend_chunk or (1 << 28 if p.name == "scientific" else 1 << 26)
        log(f"extension: {rows.nnz} + {cols.nnz} cells outside the template; filling pinned chunks")
        ext = StreamedExtension(p.m, p.n, p.I, p.J, rows, cols, max_entries, prefill=True)
        n_row, n_col = rows.nnz, cols.nnz
        chunks = [ext.bounds[0].size - 1, ext.bounds[1].size - 1]
        largest = max(ext._largest(ph, b) for ph, b in zip((rows, cols), ext.bounds))
        run = lambda: ext.run(T, P, Q, opts, col_opts)[3]  # noqa: E731
        source = (f"streamed from pinned host memory, chunks of at most {max_entries} cells "
                  f"(generated outside the timed region in {ext.prefill_s:.0f}s)")
    else:
        ext = Extension(p.m, p.n, p.u, p.i, p.r, p.I, p.J, n_chunks=16)
        n_row, n_col = ext.rows.nnz, ext.cols.nnz
        chunks = [ext.rows.bounds.size - 1, ext.cols.bounds.size - 1]
        largest = max(c[0].numel() for c in ext.rows.chunks + ext.cols.chunks)
        run = lambda: ext.run(T, P, Q, opts, col_opts)[2]  # noqa: E731
        source = "16 chunks per phase from pinned host memory"
    prep_s = time.perf_counter() - t0
    run()  # warm-up (allocations, code load)
    T.set_timing(1)
    ph = run()
    tm = T.timing()
    T.set_timing(0)
    # both phases and the assembly of the full row factors between them
    t_ext = ph["row_phase_s"] + ph["assemble_s"] + ph["col_phase_s"]
    h2d_bytes = 12 * (n_row + n_col)
    rate = h2d_probe(max(1 << 20, 12 * largest))
    copies, compute = tm["ext_h2d_ms"] / 1e3, tm["ext_compute_ms"] / 1e3
    overlap = (copies + compute - t_ext) / min(copies, compute) if min(copies, compute) > 0 else None
    log(f"extension: {n_row} + {n_col} cells in {t_ext:.4f}s (copies {copies:.3f}s, compute {compute:.3f}s)")
    return {
        "metric": "extension entries/s (row phase, assembly of the row factors, column phase)",
        "value": (n_row + n_col) / t_ext,
        "unit": "entries/s",
        "n_gpus": 1,
        "higher_is_better": True,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{p.name}: extension of the {p.I.size} x {p.J.size} template to "
                               f"{p.m} x {p.n}, {how}, fixed factors fp32, {source}",
                   "solver": args.extend_solver,
                   "row_phase_cells": n_row, "col_phase_cells": n_col,
                   "row_chunks": chunks[0], "col_chunks": chunks[1]},
        "row_phase_s": ph["row_phase_s"],
        "col_phase_s": ph["col_phase_s"],
        "assemble_s": ph["assemble_s"],
        "host_prep_s": prep_s,
        "pcie": {"h2d_bytes": h2d_bytes, "pinned_h2d_GBps": round(rate / 1e9, 2),
                 "h2d_only_s": h2d_bytes / rate,
                 "frac_of_h2d_bound": round(h2d_bytes / rate / t_ext, 4),
                 "copy_stream_s": round(copies, 4), "compute_stream_s": round(compute, 4),
                 "overlap": None if overlap is None else round(max(0.0, min(1.0, overlap)), 4)},
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the multi-GPU design is described but not built).", file=sys.stderr)
        return 2
    if args.copy_probe:
        return copy_probe()
    import torch

    import paper_2608_00977_amd as tsid
    import tsid_synth

    log(f"generating {args.config}")
    t0 = time.perf_counter()
    p = tsid_synth.make_cached(args.config, os.environ.get("TSID_SYNTH_CACHE"))
    if args.lr is not None:
        p.lr = args.lr
    gen_s = time.perf_counter() - t0
    log(f"generated {p.nnz} training cells in {gen_s:.1f}s")

    T = tsid.Tsid(0)
    T.set_pass_kernel(args.pass_kernel)
    T.set_dense_tiles(args.dense_fill)
    T.set_row_blocks(args.row_blocks)
    if args.minibatch:  # batch steps on the item pass; the epochs' loss may use the dense tiles
        T.set_minibatch(args.minibatch, args.minibatch_seed)
        T.set_pass_kernel("item")
    u = torch.from_numpy(p.u).pin_memory()
    i = torch.from_numpy(p.i).pin_memory()
    r = torch.from_numpy(p.r).pin_memory()
    t0 = time.perf_counter()
    T.build_template(p.m, p.n, u.numpy(), i.numpy(), r.numpy(), p.I, p.J, p.k)
    build_s = time.perf_counter() - t0
    info = T.info()
    nnz = info["nnz"]
    log(f"template {info['m_t']} x {info['n_t']}, |Omega*| = {nnz}, build {build_s:.3f}s")

    sim = None
    if args.similarity > 0:
        sr, sc, sv = tsid_synth.similarity_graph(p.J.size, 16, 7)
        T.set_similarity(sr, sc, sv, args.similarity)
        T.set_pass_kernel("item")
        sim = {"beta": args.similarity, "entries": int(sv.size), "links_per_column": 16}
    if args.clip_per_entry:
        T.set_pass_kernel("item")
        T.set_dense_tiles(0)
    P0 = torch.from_numpy(p.P0).cuda()
    Q0 = torch.from_numpy(p.Q0).cuda()
    clip = "per_entry" if args.clip_per_entry else p.clip
    mk = lambda ep: tsid.make_opts(epochs=ep, lam=p.lam, lr=p.lr, clip=clip, xi=p.xi,
                                   prec=p.prec, step=p.step)
    if args.warmup:
        P, Q = P0.clone(), Q0.clone()
        T.fit_template(P, Q, mk(args.warmup), want_loss=False)
        log("warmup done")

    # timed region: exactly `steps` epochs
    P, Q = P0.clone(), Q0.clone()
    T.set_timing(max(1, args.time_every))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    _, hist = T.fit_template(P, Q, mk(args.steps), want_loss=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    tm = T.timing()
    T.set_timing(False)
    kernels = T.pass_kernels()
    row_blocks = T.row_blocks()
    ms_per_step = wall * 1e3 / args.steps
    value = nnz / (ms_per_step / 1e3)
    log(f"{args.steps} epochs in {wall:.4f}s: {ms_per_step:.4f} ms/epoch, {value:.4e} cells/s")

    hist_T = float(hist[-1])  # L(P_T, Q_T), a sanity figure

    k = info["k"]
    m_t, n_t = info["m_t"], info["n_t"]
    # A slab pass split over several workgroups per block leaves the row
    # updates to its finishing kernel (timed as a fixup): its own launch then
    # reads the owner rows but does not write them.
    split = tm["fixup_launches"] > 0
    di = T.dense_info()
    sparse_nnz = nnz - di["cells"]
    if args.minibatch:
        # timed launches are the first batch's passes: its own cells, every
        # owner row read and written (lines without a cell keep theirs)
        bp = T.export_index("batch_ptr_r")
        sparse_nnz = int(bp[m_t] - bp[0])
    avg = [tm["pass_ms"][j] / max(1, tm["pass_launches"][j]) for j in range(2)]
    src_of = {"item": "fit.hip", "slab": "slab.hip"}
    cand = []

    def add(ms, by_fl, name, desc, src, which, kind, units):
        by_, fl_ = by_fl
        if ms > 0:
            cand.append(dict(ms=ms, by=by_, fl=fl_, name=name, desc=desc, src=src, which=which, kind=kind,
                             units=units))

    def pass_alg(side, sides=1):
        owners = (m_t if side == 0 else n_t) if sides == 1 else m_t + n_t
        by_, fl_ = algorithmic(sparse_nnz, owners, k, p.prec, sides)
        if kernels[side] == "slab" and split:  # the finishing kernel writes the owner rows
            by_ -= owners * 4 * k
        return by_, fl_

    pair = kernels[0] == kernels[1] and tm["pass_launches"][1] == 0 and tm["pass_launches"][0] > 0
    if pair:  # both passes in one launch (timed as the P pass; no Q pass launch)
        add(avg[0], pass_alg(0, 2), f"k_{kernels[0]}_pass_pair", "P and Q passes", src_of[kernels[0]], "pq_pass",
            kernels[0], ("hbm", "alu"))
    else:
        add(avg[0], pass_alg(0), f"k_{kernels[0]}_pass", "P pass", src_of[kernels[0]], "p_pass", kernels[0],
            ("hbm", "alu"))
        qname = "k_item_pass_sched" if kernels[1] == "item" and row_blocks > 1 else f"k_{kernels[1]}_pass"
        add(avg[1], pass_alg(1), qname, "Q pass" + (f" ({row_blocks} row blocks, one launch)" if row_blocks > 1
                                                    else ""), src_of[kernels[1]], "q_pass", kernels[1],
            ("hbm", "alu"))
    dense_avg = [tm["dense_ms"][j] / max(1, tm["dense_launches"][j]) for j in range(2)]
    dense_pair = bool(di["tiles"]) and tm["dense_launches"][1] == 0 and tm["dense_launches"][0] > 0
    if dense_pair:  # both sides' dense tiles in one launch (timed as the P side's)
        add(dense_avg[0], algorithmic(di["cells"], 0, k, p.prec, 2, False), "k_dense_pass_pair",
            "P and Q side dense tiles", "dense.hip", "pq_dense", "dense", ("hbm", "mfma"))
    elif di["tiles"]:
        for j in range(2):
            add(dense_avg[j], algorithmic(di["cells"], 0, k, p.prec, 1, False), "k_dense_pass",
                ["P", "Q"][j] + " side dense tiles", "dense.hip", ["p_dense", "q_dense"][j], "dense",
                ("hbm", "mfma"))
    dom = max(cand, key=lambda c: c["ms"])
    bound, achieved, fracs = roofline_of(dom["ms"], dom["by"], dom["fl"], dom["units"])
    src = open(os.path.join(ROOT, "paper_2608_00977_amd", "csrc", dom["src"]), "rb").read()
    sha = hashlib.sha256(src).hexdigest()
    variant = (f":minibatch{args.minibatch}" if args.minibatch else "") + (":clip2" if args.clip_per_entry else "") \
        + (":similarity" if args.similarity > 0 else "") + (f":rowblocks{row_blocks}" if row_blocks > 1 else "")
    traffic = traffic_from_profiles(sha, f"{args.config}:{dom['which']}:{dom['kind']}" + variant)
    roofline = {"bound": bound, "achieved": round(achieved, 2), "peak": PEAK[bound][0], "unit": PEAK[bound][1],
                "frac": round(fracs[bound], 4), "traffic": traffic,
                "kernel": f"{dom['name']} ({dom['desc']})",
                "bytes_per_launch": dom["by"], "flops_per_launch": dom["fl"], "avg_launch_ms": round(dom["ms"], 5),
                "fracs": {u: round(f, 4) for u, f in fracs.items()}}
    launches = [{"kernel": f"{c['name']} ({c['desc']})", "avg_launch_ms": round(c["ms"], 5),
                 "bytes_per_launch": c["by"], "flops_per_launch": c["fl"],
                 "fracs": {u: round(f, 4) for u, f in roofline_of(c["ms"], c["by"], c["fl"], c["units"])[2].items()}}
                for c in cand]
    epoch_by, epoch_fl = algorithmic(nnz, m_t + n_t, k, p.prec, 2)
    dense = None
    if di["tiles"]:
        dense = {"cells": di["cells"], "tiles": di["tiles"], "stripes": di["stripes"],
                 "share_of_cells": round(di["cells"] / max(1, nnz), 4),
                 "matrix_core_TFLOPs_issued": [round(6 * 256 * k * di["tiles"] / (c["ms"] / 1e3) / 1e12, 2)
                                               for c in cand if c["kind"] == "dense"]}

    cpu = None
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        cpu = cpu_baseline(p, args.cpu_seconds, args.minibatch, args.minibatch_seed)
        log(f"oracle {cpu['value']:.4e} cells/s over {cpu['seconds']:.1f}s")

    workload = {
        "scientific": "Scientific template fit: 16,384 x 16,384 uniform template of a 200,000 x "
                      "200,000 rank-32 matrix (10% observed), k=32, fp32, degree step",
        "rating": "Rating-shaped template fit: 65,536 x 8,192 most-observed template of a "
                  "480,189 x 17,770 Zipf matrix (100M ratings), k=64, bf16 + clip, degree step",
        "billion": "Billion-scale template fit: 1,000,000 x 100,000 most-popular template of a "
                   "10M x 1M Zipf(1.0) matrix (1e9 cells), k=128, bf16 + clip, degree step",
        "mid": "Mid template fit: 4,096 x 2,048 of 20,000 x 10,000 (2M cells), k=32, fp32",
        "tiny": "Tiny template fit: 200 x 160 of 1,000 x 800 (40k cells), k=8, fp32",
    }[args.config]
    if args.clip_per_entry:
        workload += "; clip in the per-entry order"
    if sim:
        workload += f"; multi-view term, beta {args.similarity}, {sim['entries']:,} similarity entries"
    if args.minibatch:
        workload += f"; mini-batch epochs, {args.minibatch} batches (seed {args.minibatch_seed}), loss pass each epoch"
    line = {
        "metric": "observed entries/sec per template-fit epoch; achieved HBM GB/s vs peak",
        "value": value,
        "unit": "entries/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if p.prec == "bf16" else "f32",
        "data": "synthetic (seeded generator standing in for the paper's datasets)",
        "config": {"workload": workload, "config": args.config, "m": p.m, "n": p.n,
                   "m_t": m_t, "n_t": n_t, "template_cells_train": nnz, "k": k,
                   "precision": p.prec, "step": p.step, "lr": p.lr, "lambda": p.lam,
                   "clip": clip, "parallelism": "single GPU", "similarity": sim,
                   "pass_kernels": {"p_pass": kernels[0], "q_pass": kernels[1]},
                   "q_pass_row_blocks": row_blocks,
                   "dense_tiles": dense,
                   "minibatch": {"batches": args.minibatch, "seed": args.minibatch_seed,
                                 "first_batch_cells": sparse_nnz} if args.minibatch else None},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "epoch_algorithmic": {"bytes": epoch_by, "flops": epoch_fl,
                              "GBps": round(epoch_by / (ms_per_step / 1e3) / 1e9, 2),
                              "TFLOPs": round(epoch_fl / (ms_per_step / 1e3) / 1e12, 3)},
        "launches": launches,
        "device_epoch_ms": tm["epoch_ms"] / max(1, tm["epochs"]),
        "timed_epochs": tm["epochs"],
        "kernel_ms_per_epoch": {**({"pq_pass": avg[0]} if pair else {"p_pass": avg[0], "q_pass": avg[1]}),
                                **({"pq_dense": dense_avg[0]} if dense_pair else
                                   {"p_dense": dense_avg[0], "q_dense": dense_avg[1]}),
                                "fixups": tm["fixup_ms"] / max(1, tm["epochs"]),
                                "loss_reduce": tm["reduce_ms"] / max(1, tm["reduce_launches"]) / 16},
        "loss_first_epoch": float(hist[0]),
        "build_s": build_s,
        "loss_after_timed_epochs": hist_T,
    }
    print(json.dumps(line), flush=True)
    if args.extend:
        print(json.dumps(extension_line(args, p, T, P, Q)), flush=True)
    T.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
