"""Write the full-size oracle references used by tests/test_gpu_fullsize.py.

Runs only the CPU oracle (oracle/) on the seeded synthetic workloads 1-4 at their full sizes
and stores compact JSON (objective, bias, iterations, SV counts, the first 1000 selections
with their runner-up gaps, and decision values on the first test points).  Takes several
minutes on 8 cores; rerun whenever the generator or the oracle's arithmetic changes:

    python tests/golden/make_oracle_refs.py [workload ids...]
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import oracle  # noqa: E402
from paper_2311_14908_amd import synth  # noqa: E402

N_TEST_BINARY = 256
N_TEST_OVO = 128
TRACE = 1000


def digest(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


def binary(cid: int) -> dict:
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid)
    t0 = time.time()
    # full fp64 Gram when it fits 24 GiB, else a least-recently-used set of rows
    r = oracle.train(X, y, wl.C, wl.gamma, wl.tol, cache_bytes=24 << 30, trace_len=TRACE)
    dec = oracle.decision(X, y, r.alpha, r.b, Xt[:N_TEST_BINARY], wl.gamma)
    sec = time.time() - t0
    return {
        "workload": wl.name, "n": int(X.shape[0]), "d": int(X.shape[1]), "C": wl.C, "gamma": wl.gamma,
        "tol": wl.tol, "inputs_sha256": digest(X, y, Xt[:N_TEST_BINARY]), "status": r.status,
        "iterations": r.iterations, "dual_obj": r.dual_obj, "b": r.b, "b_up": r.b_up, "b_low": r.b_low,
        "n_sv": r.n_sv, "n_bound": r.n_bound, "oracle_seconds": sec,
        "trace_ul": r.trace_ul.tolist(), "trace_gap_min": np.min(r.trace_gap, axis=1).tolist(),
        "test_decisions": dec.tolist(),
    }


def ovo() -> dict:
    wl = synth.workload(4)
    X, lab, Xt, _ = synth.generate(4)
    k = wl.classes
    t0 = time.time()
    models = oracle.train_ovo(X, lab, k, wl.C, wl.gamma, wl.tol, cache_bytes=256 << 20)
    dec, pred = oracle.predict_ovo(X, lab, k, models, Xt[:N_TEST_OVO], wl.gamma)
    sec = time.time() - t0
    return {
        "workload": wl.name, "n": int(X.shape[0]), "d": int(X.shape[1]), "k": k, "C": wl.C, "gamma": wl.gamma,
        "tol": wl.tol, "inputs_sha256": digest(X, lab, Xt[:N_TEST_OVO]), "oracle_seconds": sec,
        "pairs": [{"iterations": r.iterations, "dual_obj": r.dual_obj, "b": r.b, "n_sv": r.n_sv, "status": r.status}
                  for (_, _, r) in models],
        "test_decisions": dec.tolist(), "test_pred": pred.tolist(),
    }


def main(ids):
    for cid in ids:
        t0 = time.time()
        ref = ovo() if cid == 4 else binary(cid)
        ref["_source"] = ("fp64 CPU oracle (oracle/svm_oracle.c) on the seeded synthetic workload; written by "
                          "tests/golden/make_oracle_refs.py")
        path = os.path.join(HERE, f"oracle_full_w{cid}.json")
        with open(path, "w") as fh:
            json.dump(ref, fh, separators=(",", ":"))
        print(f"workload {cid}: {time.time() - t0:.1f} s -> {path}", flush=True)


if __name__ == "__main__":
    main([int(a) for a in sys.argv[1:]] or [1, 2, 3, 4])
