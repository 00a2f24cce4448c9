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

Default workload: the Scientific configuration's template -- 200,000 x
200,000 rank-32 ground truth, 10 % uniform observation, a 16,384 x 16,384
uniform template (about 24 M training cells), k = 32, fp32, degree step.
--config rating runs the Netflix-shaped template (65,536 x 8,192, k = 64,
bf16 factors with fp32 accumulation and clipping); --config billion the
Billion-scale template (1,000,000 x 100,000 of a 10 M x 1 M Zipf matrix,
about 4.2e8 training cells, k = 128, bf16 + clipping; its input takes a few
minutes to generate); mid / tiny are small.

Roofline: the dominant kernel is the longer of the P and Q passes (the slab
pass on evenly spread fp32 templates such as Scientific, else the item pass;
the library launches the two passes of an epoch as one kernel,
k_slab_pass_pair or k_item_pass_pair, priced with both passes' bytes, except
when the Q pass runs in row blocks),
timed with HIP events attached to its dispatches on the library's compute
stream during the timed region (every --time-every-th epoch: a timed dispatch
costs a few microseconds of wall time, which would otherwise slow the
throughput being measured); its algorithmic bytes per launch are the compulsory bytes of one
pass: the bucketed cell stream (8 B per cell), the bucket pointers (8 B per
bucket), the owner rows read and written once and the gathered rows read once
(4 B per coordinate in fp32; 2 B for bf16 copies).  A slab pass whose row
blocks are split over several workgroups leaves the row updates (the
owner-row writes) to a finishing kernel, timed with the fixups; its bytes
exclude them.

CPU baseline: the fp64 oracle (serial C) on a bounded sample of the same
template cells, for as many epochs as fit in about --cpu-seconds.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--config", default="scientific", choices=["scientific", "rating", "billion", "mid", "tiny"])
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
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--extend", action="store_true",
                    help="after the timed fit, time the end-to-end extension (row phase, then "
                         "column phase, 16 chunks each, streamed from pinned host memory) and print "
                         "a second JSON line; needs a workload with the whole matrix drawn "
                         "(rating, mid, tiny)")
    ap.add_argument("--extend-steps", type=int, default=20)
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


def pass_bytes(nnz, owners, others, k, prec, no_owner_write=False):
    """Compulsory bytes of one pass launch (see the module docstring)."""
    fb = 4 * k
    b = 8 * nnz + 8 * (owners + 1) + 2 * fb * owners + (2 * k if prec == "bf16" else fb) * others
    if prec == "bf16":
        b += 2 * k * owners  # bf16 copy of the updated rows
    if no_owner_write:
        b -= fb * owners
    return b


def dense_bytes(tiles, stripes_own, stripes_other, k):
    """Compulsory bytes of one dense-tile launch: the tile values (fp32, 1 KiB
    per tile), the tile list (4 B per tile and stripe), the owner rows of the
    stripes holding a tile read once as bf16 copies and their fp32 gradient
    sums written once, the other rows those tiles touch read once (bf16)."""
    return (1024 + 4) * tiles + 4 * stripes_own + 16 * stripes_own * (2 * k + 4 * k) \
        + 16 * stripes_other * 2 * k


def dense_flops(tiles, k):
    """Matrix-core flops of one dense-tile launch: per tile the 16 x 16 x k
    product of the residuals and the two 16 x 16 x k products of the
    gradient (high and low bf16 parts of the residual)."""
    return 3 * 2 * 256 * k * tiles


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
    import numpy as np

    import oracle
    st, rm, cm = oracle.template_maps(p.m, p.n, p.I, p.J)
    a, b, v = oracle.filter_template(p.u, p.i, p.r, rm, cm)
    S = int(min(a.size, 2_000_000))
    a, b, v = a[:S], b[:S], v[:S]
    if batches:
        run = lambda ep: oracle.fit_minibatch(a, b, v, p.P0, p.Q0, ep, p.lam, p.lr, p.step, p.clip, p.xi,
                                              bf16=p.prec == "bf16", n_batches=batches, seed=seed)
    else:
        run = lambda ep: oracle.fit(a, b, v, p.P0, p.Q0, ep, p.lam, p.lr, p.step, p.clip, p.xi,
                                    bf16=p.prec == "bf16")
    t0 = time.perf_counter()
    run(1)
    one = time.perf_counter() - t0
    epochs = max(1, int(seconds / max(one, 1e-3)))
    t0 = time.perf_counter()
    run(epochs)
    el = time.perf_counter() - t0
    return {"value": S * epochs / el, "unit": "entries/s", "cores": 1, "kind": "oracle",
            "sample": f"first {S} template cells (input order, i.e. a uniform random sample) of "
                      f"the same workload, all {p.I.size} x {p.J.size} template factor rows, "
                      f"{epochs} " + (f"mini-batch epochs ({batches} batches)" if batches else
                                      "full-gradient epochs") + ", serial fp64 C",
            "seconds": el, "nproc": os.cpu_count()}


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
    import paper_2608_00977_amd as tsid
    from paper_2608_00977_amd.extension import Extension
    if p.extra.get("omega_scope") == "template block only":
        raise SystemExit("--extend needs a workload whose whole matrix is drawn (rating, mid, tiny)")
    t0 = time.perf_counter()
    ext = Extension(p.m, p.n, p.u, p.i, p.r, p.I, p.J, n_chunks=16)
    prep_s = time.perf_counter() - t0
    col_opts = None
    if args.extend_solver == "ridge":
        opts = float(p.lam)  # exact solve per free row
        how = f"exact ridge solve per free row (lambda {p.lam}, fp64 Gram + Cholesky)"
    elif args.extend_solver == "adam":
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
    ext.run(T, P, Q, opts, col_opts)  # warm-up (allocations, code load)
    _, _, ph = ext.run(T, P, Q, opts, col_opts)
    n_row, n_col = ext.rows.nnz, ext.cols.nnz
    t_ext = ph["row_phase_s"] + ph["col_phase_s"]
    h2d_bytes = 12 * (n_row + n_col)
    rate = h2d_probe(max(1 << 20, 12 * max(c[0].numel() for c in ext.rows.chunks + ext.cols.chunks)))
    log(f"extension: {n_row} + {n_col} cells in {t_ext:.4f}s")
    return {
        "metric": "extension entries/s (row phase + column phase)",
        "value": (n_row + n_col) / t_ext,
        "unit": "entries/s",
        "n_gpus": 1,
        "higher_is_better": True,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{p.name}: extension of the {p.I.size} x {p.J.size} template to "
                               f"{p.m} x {p.n}, 16 chunks per phase, {how}, fixed factors fp32",
                   "solver": args.extend_solver,
                   "row_phase_cells": n_row, "col_phase_cells": n_col,
                   "row_chunks": ext.rows.bounds.size - 1, "col_chunks": ext.cols.bounds.size - 1},
        "row_phase_s": ph["row_phase_s"],
        "col_phase_s": ph["col_phase_s"],
        "assemble_s": ph["assemble_s"],
        "host_prep_s": prep_s,
        "pcie": {"h2d_bytes": h2d_bytes, "pinned_h2d_GBps": round(rate / 1e9, 2),
                 "h2d_only_s": h2d_bytes / rate,
                 "frac_of_h2d_bound": round(h2d_bytes / rate / t_ext, 4)},
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
    # does not write the owner rows.
    split = tm["fixup_launches"] > 0
    di = T.dense_info()
    sparse_nnz = nnz - di["cells"]
    if args.minibatch:
        # timed launches are the first batch's passes: its own cells, every
        # owner row read and written (lines without a cell keep theirs)
        bp = T.export_index("batch_ptr_r")
        sparse_nnz = int(bp[m_t] - bp[0])
    by = [pass_bytes(sparse_nnz, m_t, n_t, k, p.prec, kernels[0] == "slab" and split),
          pass_bytes(sparse_nnz, n_t, m_t, k, p.prec, kernels[1] == "slab" and split)]
    if di["tiles"]:
        # with dense tiles the item pass also reads the full bucket pointers
        # (degrees) and the tile sums of the rows in stripes holding a tile
        for j, own in ((0, m_t), (1, n_t)):
            by[j] += 8 * (own + 1) + 4 * k * min(own, 16 * di["stripes"][j])
    avg = [tm["pass_ms"][j] / max(1, tm["pass_launches"][j]) for j in range(2)]
    cand = [(avg[0], by[0], {"item": "k_item_pass", "slab": "k_slab_pass"}[kernels[0]], "P pass",
             {"item": "fit.hip", "slab": "slab.hip"}[kernels[0]], "p_pass", kernels[0]),
            (avg[1], by[1], {"item": "k_item_pass", "slab": "k_slab_pass"}[kernels[1]], "Q pass",
             {"item": "fit.hip", "slab": "slab.hip"}[kernels[1]], "q_pass", kernels[1])]
    # both passes in one launch (timed as the P pass; no Q pass launch)
    pair = kernels[0] == kernels[1] and tm["pass_launches"][1] == 0 and tm["pass_launches"][0] > 0
    if pair:
        cand = [(avg[0], by[0] + by[1], f"k_{kernels[0]}_pass_pair", "P and Q passes",
                 {"item": "fit.hip", "slab": "slab.hip"}[kernels[0]], "pq_pass", kernels[0])]
    dense_avg = [tm["dense_ms"][j] / max(1, tm["dense_launches"][j]) for j in range(2)]
    dcand = []
    # both sides' dense tiles in one launch (timed as the P side's)
    dense_pair = di["tiles"] and tm["dense_launches"][1] == 0 and tm["dense_launches"][0] > 0
    if dense_pair:
        dcand.append((dense_avg[0], sum(dense_bytes(di["tiles"], di["stripes"][j], di["stripes"][1 - j], k)
                                        for j in range(2)),
                      "k_dense_pass_pair", "P and Q side dense tiles", "dense.hip", "pq_dense", "dense"))
    elif di["tiles"]:
        for j in range(2):
            dcand.append((dense_avg[j], dense_bytes(di["tiles"], di["stripes"][j], di["stripes"][1 - j], k),
                          "k_dense_pass", ["P", "Q"][j] + " side dense tiles", "dense.hip",
                          ["p_dense", "q_dense"][j], "dense"))
    cand += dcand
    dom_ms, dom_by, kname, kside, ksrc, which, kkind = max(cand, key=lambda c: c[0])
    achieved = dom_by / (dom_ms / 1e3) / 1e9
    src = open(os.path.join(ROOT, "paper_2608_00977_amd", "csrc", ksrc), "rb").read()
    sha = hashlib.sha256(src).hexdigest()
    variant = (f":minibatch{args.minibatch}" if args.minibatch else "") + (":clip2" if args.clip_per_entry else "") \
        + (":similarity" if args.similarity > 0 else "") + (f":rowblocks{row_blocks}" if row_blocks > 1 else "")
    traffic = traffic_from_profiles(sha, f"{args.config}:{which}:{kkind}" + variant)
    epoch_bytes = by[0] + by[1] + sum(c[1] for c in dcand)
    roofline = {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBPS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                "kernel": f"{kname} ({kside})",
                "bytes_per_launch": dom_by, "avg_launch_ms": round(dom_ms, 5)}
    dense = None
    if di["tiles"]:
        fl = dense_flops(di["tiles"], k)
        dense = {"cells": di["cells"], "tiles": di["tiles"], "stripes": di["stripes"],
                 "share_of_cells": round(di["cells"] / max(1, nnz), 4),
                 "flops_per_launch": fl,
                 "mfma_TFLOPs": [round(fl * (2 if dense_pair else 1) / (c[0] / 1e3) / 1e12, 2) if c[0] else None
                                 for c in dcand],
                 "bytes_per_launch": [c[1] for c in dcand], "launches_per_epoch": len(dcand)}

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
        "compulsory_GBps_per_epoch": round(epoch_bytes / (ms_per_step / 1e3) / 1e9, 2),
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
