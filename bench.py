#!/usr/bin/env python3
"""Benchmark of kernel-SVM training by SMO (maximal violating pair) on one MI355X.

One step is one pass of the whole hot path over one synthetic workload: RBF Gram build
(MFMA), the SMO solve to tol, the finalize reduction, and decision values for the test
split.  Inputs are resident in HBM before the timed region starts.  The default workload is
the largest single-GPU binary one, 100,000 x 32 with its 40 GB fp32 Gram resident in HBM, and
the solve takes the library's automatic schedule (svm_options.working_set = -1: working-set
rounds of maximal-violating-pair steps where they beat one pair a step, decided after 128
rounds; ``schedule`` says which ran).

Prints ONE JSON line.  ``value`` is SMO iterations (pair steps) per second over the timed steps;
``train_seconds`` is the mean svm_train wall time.  ``roofline`` describes the dominant
kernel (the solver that ran) against the HBM roofline with its algorithmic bytes: per SMO step
of the per-step solver two kernel rows 8n, f read+write 16n, status n = 25n bytes; for the
working-set rounds 8n per pair step (the rows its f update needs) and 17n per round.
``pair_solver`` times the per-step solver on the same problem, with its roofline.  ``gram_build``
reports the Gram precompute against its roofline: the method's n^2 d flops at the dense fp16
MFMA peak (its contraction runs as split-fp16 products) or its 4 n^2 bytes of stores at the HBM
peak, whichever takes longer.  ``row_path`` reports the 20,000 x 784
solve with kernel rows evaluated from X at every step (4nd + 21n bytes a step), and
``row_path_large`` the same recipe at 300,000 x 784.  ``ovo`` trains the 10-class one-vs-one
workload end to end, with rooflines for its global Gram and for the launch that advances all
45 pairs; ``ovo_row_path`` runs the 45 pairs on the row path for a fixed number of steps
(4 n_p d + 21 n_p bytes per pair step).  ``paper_shapes`` times single trainings at the
shapes of the paper's own runs (102 features, 200-800 samples per class, binary and nine-class
one-vs-one) for context.  ``workloads`` trains the other binary workloads end to end once
each.  ``working_set`` trains the Gram-path workloads with the working-set solver
(svm_options.working_set = q: rounds of pair steps on q samples, f updated once a round) beside
the pair solver, and the 20,000 x 784 workload once more without a Gram (row path); its
iterations are pair steps too.  ``second_order`` trains the same three workloads with the
second-order choice of the pair's second index beside the maximal violating pair.  ``cpu_baseline`` times the fp64 CPU oracle on the same problem
on this host's cores: the whole training when it fits the time budget, else its first steps.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HBM_PEAK_GBPS = 8000.0
FP32_MFMA_PEAK_TFLOPS = 157.3
FP16_MFMA_PEAK_TFLOPS = 2500.0
ROOT = os.path.dirname(os.path.abspath(__file__))
SOLVER_SOURCES = ("paper_2311_14908_amd/csrc/smo.hip", "paper_2311_14908_amd/csrc/rbf_rows.hpp",
                  "paper_2311_14908_amd/csrc/solver_params.hpp", "paper_2311_14908_amd/csrc/pair_step.hpp")
WS_SOURCES = ("paper_2311_14908_amd/csrc/ws_smo.hip", "paper_2311_14908_amd/csrc/ws_record.hpp",
              "paper_2311_14908_amd/csrc/solver_params.hpp", "paper_2311_14908_amd/csrc/pair_step.hpp",
              "paper_2311_14908_amd/csrc/common.hpp")


def counters_path(n, d):
    return os.path.join(ROOT, "profiles", f"smo_solve_n{n}_d{d}_hbm_counters.md")


def counter_bytes_per_step(workload_name, n, d):
    """HBM bytes per SMO step measured with rocprofv3 FETCH_SIZE/WRITE_SIZE (scaled by a copy of
    known size), as recorded in profiles/; None when missing, for another workload, or when the
    solver sources changed after the counters were taken."""
    import hashlib
    try:
        line = [l for l in open(counters_path(n, d)) if "solver_sources_sha256" in l][0]
        rec = json.loads(line.strip())
    except (OSError, IndexError, ValueError):
        return None
    h = hashlib.sha256()
    for p in SOLVER_SOURCES:
        h.update(open(os.path.join(ROOT, p), "rb").read())
    if rec.get("solver_sources_sha256") != h.hexdigest() or rec.get("workload") != workload_name:
        return None
    return rec


def ws_counter_bytes(workload_name, n, d):
    """HBM bytes per working-set round from rocprofv3 FETCH_SIZE/WRITE_SIZE, as recorded in
    profiles/ for the working-set solver; None when missing, for another workload, or stale."""
    import hashlib
    try:
        path = os.path.join(ROOT, "profiles", f"ws_solve_n{n}_d{d}_hbm_counters.md")
        line = [l for l in open(path) if "ws_sources_sha256" in l][0]
        rec = json.loads(line.strip())
    except (OSError, IndexError, ValueError):
        return None
    h = hashlib.sha256()
    for p in WS_SOURCES:
        h.update(open(os.path.join(ROOT, p), "rb").read())
    if rec.get("ws_sources_sha256") != h.hexdigest() or rec.get("workload") != workload_name:
        return None
    return rec


def gram_roofline(n, d, seconds):
    """The Gram precompute against its roofline: the method's n^2 d flops (symmetric count) at the
    dense fp16 MFMA peak (the contraction runs as split-fp16 products on the fp16 instruction)
    against its 4 n^2 bytes of stores at the HBM peak; `bound` is the resource whose ideal time is
    longer, and achieved/peak/frac are given for it (both fractions are reported)."""
    flops = float(n) * n * d
    wbytes = 4.0 * n * n
    tf = flops / seconds / 1e12 if seconds > 0 else None
    gbps = wbytes / seconds / 1e9 if seconds > 0 else None
    t_mfma, t_hbm = flops / (FP16_MFMA_PEAK_TFLOPS * 1e12), wbytes / (HBM_PEAK_GBPS * 1e9)
    mfma = {"achieved": tf, "peak": FP16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": tf / FP16_MFMA_PEAK_TFLOPS if tf else None}
    hbm = {"achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": gbps / HBM_PEAK_GBPS if gbps else None}
    bound = "mfma" if t_mfma >= t_hbm else "hbm"
    return {"kernel": "gram_rbf_f16x3 (fp32 inputs split into fp16 halves, 3 products per fp32 product)",
            "bound": bound, **(mfma if bound == "mfma" else hbm), "flops": flops, "gram_bytes": wbytes,
            "seconds": seconds, "ideal_seconds": {"mfma": t_mfma, "hbm_write": t_hbm},
            "mfma_frac": mfma["frac"], "hbm_write_frac": hbm["frac"],
            "executed_fp16_tflops": 3.0 * tf if tf else None,
            "fp32_equivalent_vs_fp32_mfma_peak": tf / FP32_MFMA_PEAK_TFLOPS if tf else None}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=3, help="synthetic workload id (0..3 binary)")
    ap.add_argument("--gram", choices=["auto", "on", "off"], default="auto")
    ap.add_argument("--working-set", type=int, default=-1,
                    help="svm_options.working_set of the timed trainings: -1 = automatic (rounds where they "
                         "beat the per-step solver, decided after 128 rounds), 0 = per-step solver, q = rounds of q")
    ap.add_argument("--row-path-steps", type=int, default=4000, help="SMO steps of the row-path measurement (0 = skip)")
    ap.add_argument("--row-large-n", type=int, default=300_000,
                    help="samples of the large row-path measurement (workload 1's recipe, X far larger than the "
                         "on-chip memories and the Infinity Cache; 0 = skip)")
    ap.add_argument("--row-large-steps", type=int, default=200, help="SMO steps of the large row-path measurement")
    ap.add_argument("--cpu-seconds", type=float, default=45.0,
                    help="CPU-oracle time budget: the whole training when its predicted time fits, else the first "
                         "steps that fit (0 = skip)")
    ap.add_argument("--no-ovo", action="store_true", help="skip the one-vs-one measurement (60000x784, 10 classes)")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the end-to-end trainings of the other binary workloads")
    ap.add_argument("--ws-q", type=str, default="32,128",
                    help="working-set sizes of the working-set leg, comma separated ('' = skip)")
    ap.add_argument("--no-second-order", action="store_true",
                    help="skip the second-order selection leg (Gram-path binary workloads)")
    ap.add_argument("--no-paper-shapes", action="store_true",
                    help="skip the context runs at the paper's shapes (d=102, 200-800 per class)")
    ap.add_argument("--ovo-row-steps", type=int, default=300,
                    help="SMO steps per pair of the one-vs-one row-path measurement (0 = skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="first run one plain device-to-device copy of BYTES (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2311_14908_amd import svmx, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    svmx.load()
    if args.copy_calibration > 0:
        src = torch.ones(args.copy_calibration // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()
    wl = synth.workload(args.workload)
    if wl.classes != 2:
        print("bench.py times the binary workloads (0..3)", file=sys.stderr)
        sys.exit(2)
    gram_mode = {"auto": svmx.GRAM_AUTO, "on": svmx.GRAM_ON, "off": svmx.GRAM_OFF}[args.gram]
    X, y, Xt, yt = synth.generate(args.workload)
    n, d = X.shape
    m = Xt.shape[0]
    Xd, yd, Xtd = (torch.from_numpy(a).cuda() for a in (X, y, Xt))
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    def step():
        out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram_mode, working_set=args.working_set)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        dec = svmx.svm_predict(Xd, yd, out.alpha, out.b, wl.gamma, Xtd)
        e1.record(stream)
        return out, dec, (e0, e1)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    runs = [step() for _ in range(args.steps)]
    torch.cuda.synchronize()
    T = time.perf_counter() - t0

    st = [r[0].stats for r in runs]
    iters = sum(s["iterations"] for s in st)
    t_pred = [r[2][0].elapsed_time(r[2][1]) * 1e-3 for r in runs]
    mean = lambda k: float(np.mean([s[k] for s in st]))
    dec = runs[-1][1].cpu().numpy()
    acc = float(np.mean(np.where(dec > 0, 1, -1) == yt))
    launches = sum(s["launches"] for s in st)
    t_kernel = sum(s["t_kernel"] for s in st)
    rounds = sum(s["rounds"] for s in st)
    schedule = st[0]["schedule"]
    gram_used = bool(st[0]["gram_used"])
    if schedule == 1:
        # working-set rounds: per pair step two kernel rows (8n, the rows the f update needs), per
        # round f read and written and the status (17n)
        solver_bytes = 8.0 * n * iters + 17.0 * n * rounds
        kname = "ws_solve"
        counters = ws_counter_bytes(wl.name, n, d)
        traffic = counters["ws_solve_hbm_bytes_per_round"] * rounds / launches if counters else None
        note = ("working-set rounds: bound by the latency of the round's chain (own lists, two merge levels, "
                "K_BB, the pair steps in one wave, the f update), not by HBM bandwidth")
    else:
        # per-step solver: two kernel rows 8n, f read+write 16n, status n per SMO step
        solver_bytes = 25.0 * n * iters
        kname = "smo_solve"
        counters = counter_bytes_per_step(wl.name, n, d)
        traffic = (counters["gram_path_hbm_bytes_per_smo_step"] * iters / launches
                   if counters and gram_used else None)
        note = ("a step moves 25n algorithmic bytes but is bound by latency: the cross-workgroup exchange of the "
                "selections and the dependent read of the two Gram rows")
    solver_gbps = solver_bytes / t_kernel / 1e9

    result = {
        "metric": "SMO iterations/sec + train seconds; kernel-row HBM GB/s vs peak",
        "value": iters / T,
        "unit": "SMO iterations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * T / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 kernel values (Gram contraction: split-fp16 x3 MFMA products, fp32 accumulation), f64 solve",
        "data": "synthetic (seeded), resident in HBM",
        "config": {"workload": f"{wl.name}: binary RBF-SVM, C={wl.C:g}, gamma={wl.gamma:g}, tol={wl.tol:g}",
                   "n": n, "d": d, "m_test": m, "gram": bool(st[0]["gram_used"]), "working_set": args.working_set},
        "train_seconds": mean("t_total"),
        "iterations_per_step": iters / args.steps,
        "phases_s": {"upload": mean("t_upload"), "gram": mean("t_gram"), "solve": mean("t_solve"), "solver_kernel": t_kernel / args.steps,
                     "finalize": mean("t_finalize"), "predict": float(np.mean(t_pred))},
        "n_sv": st[-1]["n_sv"], "n_bound_sv": st[-1]["n_bound_sv"], "dual_obj": st[-1]["dual_obj"],
        "test_accuracy": acc,
        "schedule": {0: "per-step solver", 1: "working-set rounds", 2: "working-set probe, then per-step solver"}[schedule],
        "working_set_rounds": rounds / args.steps,
        "roofline": {"kernel": kname, "bound": "hbm", "achieved": solver_gbps, "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": solver_gbps / HBM_PEAK_GBPS, "traffic": traffic,
                     "bytes": solver_bytes / launches, "bytes_per_launch_rule":
                         "8n per pair step + 17n per round" if schedule == 1 else "25n per SMO step",
                     "launch_avg_ms": 1e3 * t_kernel / launches,
                     "us_per_smo_step": 1e6 * t_kernel / iters,
                     "us_per_round": 1e6 * t_kernel / rounds if rounds else None,
                     "note": note},
        # the default Gram runs the fp32 contraction as three fp16 MFMA products per fp32 product
        # (split halves) on the fp16 MFMA instruction, so its peak is the dense fp16 one; the
        # achieved rate counts the method's n^2 d flops (symmetric), not the executed products
        "gram_build": gram_roofline(n, d, mean("t_gram")),
    }

    # The same training from host arrays: X and y in pinned host memory, copied to the device,
    # trained, alpha copied back (the interface itself takes device buffers, so this is context,
    # never `value`).
    Xh = torch.empty(X.shape, dtype=torch.float32, pin_memory=True)
    yh = torch.empty(y.shape, dtype=torch.int32, pin_memory=True)
    Xh.copy_(torch.from_numpy(X))
    yh.copy_(torch.from_numpy(y))
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    Xd2, yd2 = Xh.to("cuda", non_blocking=True), yh.to("cuda", non_blocking=True)
    torch.cuda.synchronize()
    t_h2d = time.perf_counter() - t1
    t1 = time.perf_counter()
    Xd2, yd2 = Xh.to("cuda", non_blocking=True), yh.to("cuda", non_blocking=True)
    oh = svmx.svm_train(Xd2, yd2, wl.C, wl.gamma, wl.tol, gram=gram_mode, working_set=args.working_set)
    ah = oh.alpha.to("cpu")
    torch.cuda.synchronize()
    t_host = time.perf_counter() - t1
    result["host_arrays"] = {"train_seconds": t_host, "h2d_seconds": t_h2d,
                             "h2d_GBps": (X.nbytes + y.nbytes) / t_h2d / 1e9,
                             "note": "pinned host X and y copied in, trained, alpha copied out; PCIe "
                                     "included; not the headline value"}
    del Xd2, yd2, Xh, yh, ah

    # The per-step solver (one maximal violating pair a step, svm_options.working_set = 0) on the same
    # problem: the method step by step, with the roofline of its kernel.
    if args.working_set != 0:
        svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram_mode)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        pr = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram_mode)
        torch.cuda.synchronize()
        tpr = time.perf_counter() - t1
        ps_ = pr.stats
        pb = 25.0 * n * ps_["iterations"]
        pc = counter_bytes_per_step(wl.name, n, d)
        ptraffic = (pc["gram_path_hbm_bytes_per_smo_step"] * ps_["iterations"] / ps_["launches"]
                    if pc and ps_["gram_used"] else None)
        result["pair_solver"] = {"kernel": "smo_solve", "train_seconds": tpr, "smo_iterations": ps_["iterations"],
                                 "iters_per_s": ps_["iterations"] / tpr, "bound": "hbm",
                                 "achieved": pb / ps_["t_kernel"] / 1e9, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                 "frac": pb / ps_["t_kernel"] / 1e9 / HBM_PEAK_GBPS, "traffic": ptraffic,
                                 "bytes_per_step": 25.0 * n, "launch_avg_ms": 1e3 * ps_["t_kernel"] / ps_["launches"],
                                 "us_per_smo_step": 1e6 * ps_["t_kernel"] / ps_["iterations"],
                                 "dual_obj": ps_["dual_obj"]}
        del pr

    # The row path on the 20,000 x 784 workload (where the kernel-row GEMV is the step's work) and on
    # the same recipe at 300,000 x 784.
    w1 = synth.workload(1)
    counters1 = counter_bytes_per_step(w1.name, w1.n, w1.d)
    if args.row_path_steps > 0:
        k = args.row_path_steps
        X1, y1, _, _ = synth.generate(1, m=1)
        n1, d1 = X1.shape
        X1d, y1d = torch.from_numpy(X1).cuda(), torch.from_numpy(y1).cuda()
        svmx.svm_train(X1d, y1d, w1.C, w1.gamma, w1.tol, gram=svmx.GRAM_OFF, max_iter=64)
        torch.cuda.synchronize()
        rb = 4.0 * n1 * d1 + 21.0 * n1
        # default (the first rows of every workgroup's slice resident in LDS), then every row
        # streamed from HBM at every step
        for key, res, ckey in (("row_path", 0, "row_path_hbm_bytes_per_smo_step"),
                               ("row_path_streamed", -1, "row_path_streamed_hbm_bytes_per_smo_step")):
            r = svmx.svm_train(X1d, y1d, w1.C, w1.gamma, w1.tol, gram=svmx.GRAM_OFF, max_iter=k, resident_rows=res)
            s = r.stats
            gbps = rb * s["iterations"] / s["t_kernel"] / 1e9
            rtraffic = (counters1[ckey] * s["iterations"] / s["launches"] if counters1 and ckey in counters1 else None)
            result[key] = {"kernel": "smo_solve (row path)", "workload": w1.name, "bound": "hbm",
                           "smo_steps": s["iterations"], "iters_per_s": s["iterations"] / s["t_kernel"],
                           "us_per_step": 1e6 * s["t_kernel"] / s["iterations"], "bytes_per_step": rb,
                           "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": gbps / HBM_PEAK_GBPS,
                           "traffic": rtraffic, "resident_rows_per_workgroup": s["resident_rows"]}
            if res == 0:
                # at this size X stays on chip: the resident rows in LDS, the others in the L2 of
                # their XCD from step to step (traffic shows what reaches HBM)
                result[key].update({"bound": "on-chip (X in LDS and L2)",
                                    "note": "achieved counts the algorithmic bytes 4nd+21n; X is not re-read from "
                                            "HBM at this size, so frac is an effective rate, not HBM use"})
        # the HBM row cache (direct-mapped, 4096 rows): the same steps with it on
        ld1 = (n1 + 63) // 64 * 64
        rc = svmx.svm_train(X1d, y1d, w1.C, w1.gamma, w1.tol, gram=svmx.GRAM_OFF, max_iter=k,
                            row_cache_bytes=4 * ld1 * 4096)
        rcs = rc.stats
        result["row_cache"] = {"slots": 4096, "smo_steps": rcs["iterations"],
                               "us_per_step": 1e6 * rcs["t_kernel"] / rcs["iterations"],
                               "us_per_step_without": result["row_path"]["us_per_step"],
                               "note": "the maximal violating pair rarely revisits both rows of a step, so the cache "
                                       "only adds its stores; off by default"}
        del X1d, y1d

    if args.row_large_n > 0 and args.row_large_steps > 0:
        # The same recipe at a size where X (4 n d bytes) exceeds LDS, L2 and the 256 MB Infinity
        # Cache together, so every step streams most of X from HBM.
        # Drawn on the device with torch's seeded generator (workload 1's recipe; the parity tests
        # draw the same inputs).
        nl, dl = args.row_large_n, w1.d
        XLd, yLd = synth.sparse_projection_on_device(nl, dl, seed=1)
        svmx.svm_train(XLd, yLd, w1.C, w1.gamma, w1.tol, gram=svmx.GRAM_OFF, max_iter=16)
        torch.cuda.synchronize()
        r = svmx.svm_train(XLd, yLd, w1.C, w1.gamma, w1.tol, gram=svmx.GRAM_OFF, max_iter=args.row_large_steps)
        s = r.stats
        rbl = 4.0 * nl * dl + 21.0 * nl
        gbps = rbl * s["iterations"] / s["t_kernel"] / 1e9
        ckey = "row_path_large_hbm_bytes_per_smo_step"
        rtraffic = (counters1[ckey] * s["iterations"] / s["launches"] if counters1 and ckey in counters1 else None)
        result["row_path_large"] = {"kernel": "smo_solve (row path)", "bound": "hbm",
                                    "workload": f"sparse-proj-n{nl}-d{dl} (recipe of {w1.name})",
                                    "smo_steps": s["iterations"], "us_per_step": 1e6 * s["t_kernel"] / s["iterations"],
                                    "bytes_per_step": rbl, "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                    "frac": gbps / HBM_PEAK_GBPS, "traffic": rtraffic,
                                    "resident_rows_per_workgroup": s["resident_rows"]}
        del XLd, yLd
        torch.cuda.empty_cache()

    if not args.no_ovo:
        wo = synth.workload(4)
        Xo, lo, Xto, lto = synth.generate(4)
        Xod, lod, Xtod = (torch.from_numpy(a).cuda() for a in (Xo, lo, Xto))
        svmx.svm_train_ovo(Xod, lod, wo.classes, wo.C, wo.gamma, wo.tol)  # warm-up
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        oo = svmx.svm_train_ovo(Xod, lod, wo.classes, wo.C, wo.gamma, wo.tol)
        torch.cuda.synchronize()
        t_train = time.perf_counter() - t1
        t1 = time.perf_counter()
        _, pred = svmx.svm_predict_ovo(Xod, lod, wo.classes, oo.alpha, oo.b, wo.gamma, Xtod)
        torch.cuda.synchronize()
        t_pred = time.perf_counter() - t1
        it = sum(p["iterations"] for p in oo.stats)
        no = Xo.shape[0]
        _, osz = svmx.ovo_offsets(lo, wo.classes)
        # the launch that advances all 45 pairs: 25 n_p algorithmic bytes per pair step (two
        # Gram row slices, f read and write, status), over the solver kernel's time
        obytes = sum(25.0 * float(sz) * p["iterations"] for sz, p in zip(osz, oo.stats))
        otk = oo.stats[0]["t_kernel"]
        result["ovo"] = {"workload": f"{wo.name}: {wo.classes}-class one-vs-one RBF-SVM, 45 pairs, C={wo.C:g}, "
                                     f"gamma={wo.gamma:g}, tol={wo.tol:g}",
                         "train_seconds": t_train, "smo_iterations": it, "iters_per_s": it / t_train,
                         "upload_seconds": oo.stats[0]["t_upload"], "gram_seconds": oo.stats[0]["t_gram"],
                         "solver_kernel_seconds": otk, "predict_seconds": t_pred,
                         "test_accuracy": float(np.mean(pred.cpu().numpy() == lto)),
                         "gram_build": gram_roofline(no, Xo.shape[1], oo.stats[0]["t_gram"]),
                         "roofline": {"kernel": "smo_solve (Gram path, 45 pairs in one launch)", "bound": "hbm",
                                      "bytes": obytes, "bytes_per_pair_step": "25*n_p", "kernel_seconds": otk,
                                      "launches": oo.stats[0]["launches"], "achieved": obytes / otk / 1e9,
                                      "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                                      "frac": obytes / otk / 1e9 / HBM_PEAK_GBPS,
                                      "us_per_pair_step": 1e6 * otk / it * len(osz)}}
        if args.ovo_row_steps > 0:
            # the same 45 pairs on the row path: every pair evaluates its kernel rows from X at
            # every step, all pairs in one launch (batched one-vs-one steps)
            svmx.svm_train_ovo(Xod, lod, wo.classes, wo.C, wo.gamma, wo.tol, gram=svmx.GRAM_OFF, max_iter=20)
            torch.cuda.synchronize()
            orow = svmx.svm_train_ovo(Xod, lod, wo.classes, wo.C, wo.gamma, wo.tol, gram=svmx.GRAM_OFF,
                                      max_iter=args.ovo_row_steps)
            _, sizes = svmx.ovo_offsets(lo, wo.classes)
            its = [p["iterations"] for p in orow.stats]
            ob = sum(float(i) * (4.0 * m * Xo.shape[1] + 21.0 * m) for i, m in zip(its, sizes))
            tko = orow.stats[0]["t_kernel"]
            result["ovo_row_path"] = {"kernel": "smo_solve (row path, 45 pairs in one launch)",
                                      "bound": "Infinity Cache (X fits it)",
                                      "smo_steps_per_pair": [min(its), max(its)], "bytes": ob,
                                      "bytes_per_pair_step": "4*n_p*d + 21*n_p", "kernel_seconds": tko,
                                      "achieved": ob / tko / 1e9, "peak": None, "unit": "GB/s", "frac": None,
                                      "achieved_vs_hbm_peak": ob / tko / 1e9 / HBM_PEAK_GBPS,
                                      "note": "algorithmic bytes over kernel time; the class-sorted X (188 MB) "
                                              "fits the 256 MB Infinity Cache, which serves it, so the HBM peak "
                                              "does not bound this leg"}
            del orow
        del Xod, lod, Xtod, oo
        torch.cuda.empty_cache()

    if not args.no_workloads:
        # the other binary workloads, end to end (one warm-up and one timed training each)
        per = {}
        for cid in (0, 1, 2, 3):
            if cid == args.workload:
                continue
            wk = synth.workload(cid)
            Xk, yk, _, _ = synth.generate(cid, m=1)
            Xkd, ykd = torch.from_numpy(Xk).cuda(), torch.from_numpy(yk).cuda()
            svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, working_set=args.working_set)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            rk = svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, working_set=args.working_set)
            torch.cuda.synchronize()
            tk = time.perf_counter() - t1
            sk = rk.stats
            nk = Xk.shape[0]
            gb = 25.0 * nk * sk["iterations"] / sk["t_kernel"] / 1e9
            per[wk.name] = {"train_seconds": tk, "smo_iterations": sk["iterations"], "schedule": sk["schedule"],
                            "rounds": sk["rounds"],
                            "iters_per_s": sk["iterations"] / sk["t_solve"], "gram_seconds": sk["t_gram"],
                            "us_per_smo_step": 1e6 * sk["t_kernel"] / sk["iterations"], "gram_used": sk["gram_used"],
                            "solver_GBps": gb, "solver_frac_of_hbm_peak": gb / HBM_PEAK_GBPS}
            if sk["gram_used"] and nk > 4096:
                per[wk.name]["gram_build"] = gram_roofline(nk, Xk.shape[1], sk["t_gram"])
            del Xkd, ykd, rk
            torch.cuda.empty_cache()
        result["workloads"] = per

    if args.ws_q:
        # the working-set solver (rounds of pair steps on q samples, f updated once a round)
        # beside the pair solver, end to end on the Gram-path workloads: one warm-up and one
        # timed training each; iterations are pair steps, as for the pair solver
        qs = [int(v) for v in args.ws_q.split(",") if v]
        wsr = {}
        for cid in (1, 2, 3):
            wk = synth.workload(cid)
            Xk, yk, _, _ = synth.generate(cid, m=1)
            Xkd, ykd = torch.from_numpy(Xk).cuda(), torch.from_numpy(yk).cuda()
            ent = {}
            for q in [0] + qs + [-1]:
                svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, gram=svmx.GRAM_ON, working_set=q)
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                rk = svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, gram=svmx.GRAM_ON, working_set=q)
                torch.cuda.synchronize()
                tk = time.perf_counter() - t1
                sk = rk.stats
                ent["pair" if q == 0 else ("auto" if q < 0 else f"q{q}")] = {
                    "train_seconds": tk, "smo_iterations": sk["iterations"], "rounds": sk["rounds"],
                    "schedule": sk["schedule"], "us_per_round": 1e6 * sk["t_kernel"] / sk["rounds"] if sk["rounds"] else None,
                    "iters_per_s": sk["iterations"] / sk["t_solve"], "solver_kernel_seconds": sk["t_kernel"],
                    "dual_obj": sk["dual_obj"]}
                del rk
            for key, e in ent.items():
                e["speedup_vs_pair"] = ent["pair"]["train_seconds"] / e["train_seconds"]
            wsr[wk.name] = ent
            if cid == 1:
                # the same problem without a Gram: pair steps evaluate two rows of K from X a
                # step, working-set rounds evaluate K(B, .) for all of B in one pass a round
                rent = {}
                for q in [0] + [v for v in qs if v <= 128] + [-1]:
                    kw = dict(gram=svmx.GRAM_OFF, working_set=q)
                    svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, **kw)
                    torch.cuda.synchronize()
                    t1 = time.perf_counter()
                    rk = svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, **kw)
                    torch.cuda.synchronize()
                    tk = time.perf_counter() - t1
                    sk = rk.stats
                    rent["pair" if q == 0 else ("auto" if q < 0 else f"q{q}")] = {
                        "train_seconds": tk, "smo_iterations": sk["iterations"], "rounds": sk["rounds"],
                        "schedule": sk["schedule"],
                        "iters_per_s": sk["iterations"] / sk["t_solve"], "dual_obj": sk["dual_obj"]}
                    del rk
                for key, e in rent.items():
                    e["speedup_vs_pair"] = rent["pair"]["train_seconds"] / e["train_seconds"]
                wsr[wk.name + " (row path)"] = rent
            del Xkd, ykd
            torch.cuda.empty_cache()
        result["working_set"] = wsr

    if not args.no_second_order:
        # second-order choice of l (svm_options.selection) beside the maximal violating pair on
        # the Gram-path binary workloads: steps, microseconds a step, train seconds (one warm-up,
        # one timed training each)
        sor = {}
        for cid in (1, 2, 3):
            wk = synth.workload(cid)
            Xk, yk, _, _ = synth.generate(cid, m=1)
            Xkd, ykd = torch.from_numpy(Xk).cuda(), torch.from_numpy(yk).cuda()
            ent = {}
            for name, sel in (("mvp", svmx.SELECT_MVP), ("second_order", svmx.SELECT_SECOND_ORDER)):
                svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, gram=svmx.GRAM_ON, selection=sel)
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                rk = svmx.svm_train(Xkd, ykd, wk.C, wk.gamma, wk.tol, gram=svmx.GRAM_ON, selection=sel)
                torch.cuda.synchronize()
                tk = time.perf_counter() - t1
                sk = rk.stats
                ent[name] = {"train_seconds": tk, "smo_iterations": sk["iterations"],
                             "us_per_smo_step": 1e6 * sk["t_kernel"] / sk["iterations"],
                             "solver_kernel_seconds": sk["t_kernel"], "dual_obj": sk["dual_obj"]}
                del rk
            ent["second_order"]["steps_vs_mvp"] = ent["second_order"]["smo_iterations"] / ent["mvp"]["smo_iterations"]
            ent["second_order"]["speedup_vs_mvp"] = ent["mvp"]["train_seconds"] / ent["second_order"]["train_seconds"]
            sor[wk.name] = ent
            del Xkd, ykd
            torch.cuda.empty_cache()
        result["second_order"] = sor

    if not args.no_paper_shapes:
        # context runs of the paper's shapes (102 features, 200-800 samples per class; binary and
        # nine-class one-vs-one): wall seconds of one training from device-resident inputs
        ps = synth.PAPER_SHAPE
        shapes = {"binary": {}, "ovo9": {}}
        for per in (200, 400, 600, 800):
            Xp, lp = synth.paper_shaped(per, 2, seed=per)
            yp = np.where(lp == 0, 1, -1).astype(np.int32)
            Xpd, ypd = torch.from_numpy(Xp).cuda(), torch.from_numpy(yp).cuda()
            svmx.svm_train(Xpd, ypd, ps["C"], ps["gamma"], ps["tol"])
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            rp = svmx.svm_train(Xpd, ypd, ps["C"], ps["gamma"], ps["tol"])
            torch.cuda.synchronize()
            shapes["binary"][per] = {"train_seconds": time.perf_counter() - t1, "smo_iterations": rp.stats["iterations"]}
            Xp, lp = synth.paper_shaped(per, 9, seed=per)
            Xpd, lpd = torch.from_numpy(Xp).cuda(), torch.from_numpy(lp).cuda()
            svmx.svm_train_ovo(Xpd, lpd, 9, ps["C"], ps["gamma"], ps["tol"])
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            op = svmx.svm_train_ovo(Xpd, lpd, 9, ps["C"], ps["gamma"], ps["tol"])
            torch.cuda.synchronize()
            shapes["ovo9"][per] = {"train_seconds": time.perf_counter() - t1,
                                   "smo_iterations": sum(q["iterations"] for q in op.stats)}
        result["paper_shapes"] = {"d": ps["d"], "per_class": [200, 400, 600, 800], **shapes}

    if args.cpu_seconds > 0:
        # The fp64 oracle on the same problem: the whole training when its time, predicted from
        # a probe of its first steps and the GPU's step count, fits the budget; else the first
        # steps that fit.  All host threads (OpenMP over the per-sample loops).
        import oracle
        threads = oracle.max_threads()
        cache = 16 << 30  # the full fp64 Gram when it fits, else a least-recently-used row cache
        probe = 20
        t1 = time.perf_counter()
        oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=probe, cache_bytes=cache)
        rate = probe / max(time.perf_counter() - t1, 1e-6)
        expect = 1.2 * iters / args.steps
        full = expect <= rate * args.cpu_seconds
        k = None if full else int(max(probe, rate * args.cpu_seconds))
        t1 = time.perf_counter()
        r = oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=k, cache_bytes=cache)
        tc = time.perf_counter() - t1
        what = (f"the whole training ({r.iterations} SMO steps to tol, status {r.status})" if k is None
                else f"the first {r.iterations} SMO steps")
        result["cpu_baseline"] = {"value": r.iterations / tc, "unit": "SMO iterations/s", "cores": threads,
                                  "kind": "oracle", "seconds": tc,
                                  "sample": f"{what} of the same {n}x{d} problem ({wl.name}), fp64 oracle on "
                                            f"{threads} host threads, {tc:.1f} s"}
        # the same oracle on one host thread: a bounded prefix of the same problem, and the whole
        # 1,000 x 16 training
        k1 = int(max(10, rate / max(threads, 1) * args.cpu_seconds / 10))
        t1 = time.perf_counter()
        r1 = oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=k1, cache_bytes=cache, threads=1)
        t1c = time.perf_counter() - t1
        w0 = synth.workload(0)
        X0, y0, _, _ = synth.generate(0, m=1)
        t1 = time.perf_counter()
        r0 = oracle.train(X0, y0, w0.C, w0.gamma, w0.tol, threads=1)
        t0c = time.perf_counter() - t1
        result["cpu_baseline_single_thread"] = {
            "value": r1.iterations / t1c, "unit": "SMO iterations/s", "cores": 1, "kind": "oracle",
            "sample": f"first {r1.iterations} SMO steps of the same {n}x{d} problem on one thread, {t1c:.1f} s",
            "small_workload": {"workload": w0.name, "train_seconds": t0c, "smo_iterations": r0.iterations}}
    print(json.dumps(result), flush=True)
    # release the device state before the interpreter exits (nothing of the library outlives a
    # call; torch's cached blocks go back here, not in the exit handlers)
    torch.cuda.synchronize()
    del Xd, yd, Xtd, runs
    torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
