"""CPU oracle for kernel-SVM training by SMO (fp64, plain, slow).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU-baseline leg
of the benchmark may import this package; the product library never does, and the
two share no code.  The arithmetic lives in ``svm_oracle.c`` (built with gcc by
``oracle.build``); this module marshals NumPy arrays and adds the one-vs-one
orchestration, which is pure bookkeeping around the binary solver.

One-vs-one (paper, Section III.A: m classes give m(m-1)/2 independent binary
problems; Section III.B: the multiclass solve runs many binary SMOs).  Readings:
pairs (a<b) in lexicographic order; class a is +1, class b is -1; the local sample
order is the class-a samples by increasing original index, then the class-b
samples likewise; a test point votes a when d>0, else b; the predicted class is the
one with most votes, ties to the smaller class id.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np

from .build import build, lib_path

RBF, LINEAR = 0, 1


class _Res(C.Structure):
    _fields_ = [("iterations", C.c_int64), ("b", C.c_double), ("b_up", C.c_double), ("b_low", C.c_double),
                ("dual_obj", C.c_double), ("n_sv", C.c_int64), ("n_bound", C.c_int64), ("status", C.c_int32),
                ("pad", C.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(lib_path()) or os.path.getmtime(lib_path()) < os.path.getmtime(
                os.path.join(os.path.dirname(__file__), "svm_oracle.c")):
            build()
        lib = C.CDLL(lib_path())
        P = C.c_void_p
        lib.oracle_kernel_value.restype = C.c_double
        lib.oracle_kernel_value.argtypes = [P, P, C.c_int64, C.c_int, C.c_double]
        lib.oracle_kernel_rows.restype = None
        lib.oracle_kernel_rows.argtypes = [P, C.c_int64, C.c_int64, P, C.c_int64, C.c_int, C.c_double, P, C.c_int]
        lib.oracle_train.restype = C.c_int
        lib.oracle_train.argtypes = [P, P, C.c_int64, C.c_int64, C.c_int, C.c_double, C.c_double, C.c_double,
                                     C.c_int64, C.c_int64, C.c_int, P, P, C.POINTER(_Res), C.c_int64, P, P, P,
                                     C.c_int]
        lib.oracle_decision.restype = None
        lib.oracle_decision.argtypes = [P, P, P, C.c_double, C.c_int64, C.c_int64, C.c_int, C.c_double, P,
                                        C.c_int64, P, C.c_int]
        lib.oracle_f_from_alpha.restype = None
        lib.oracle_f_from_alpha.argtypes = [P, P, P, C.c_int64, C.c_int64, C.c_int, C.c_double, P, C.c_int64, P,
                                            C.c_int]
        lib.oracle_train_ws.restype = C.c_int
        lib.oracle_train_ws.argtypes = [P, P, C.c_int64, C.c_int64, C.c_int, C.c_double, C.c_double, C.c_double,
                                        C.c_int64, C.c_double, C.c_int64, C.c_int64, C.c_int64, C.c_int, P, P,
                                        C.POINTER(_Res), P, C.c_int64, P, P, P, P, C.c_int64, P]
        lib.oracle_ws_select.restype = C.c_int64
        lib.oracle_ws_select.argtypes = [P, P, P, C.c_int64, C.c_double, C.c_int64, P]
        lib.oracle_max_threads.restype = C.c_int
        lib.oracle_max_threads.argtypes = []
        _lib = lib
    return _lib


def _p(a):
    return a.ctypes.data_as(C.c_void_p)


def _f32(X):
    return np.ascontiguousarray(X, dtype=np.float32)


def max_threads() -> int:
    return int(_load().oracle_max_threads())


@dataclass
class TrainResult:
    alpha: np.ndarray
    b: float
    b_up: float
    b_low: float
    dual_obj: float
    iterations: int
    n_sv: int
    n_bound: int
    status: int
    f: np.ndarray | None = None
    trace_ul: np.ndarray | None = None   # [steps, 2] int32 (u, l)
    trace_b: np.ndarray | None = None    # [steps, 2] (b_up, b_low)
    trace_gap: np.ndarray | None = None  # [steps, 2] runner-up gaps of the two scans


MVP, SECOND_ORDER = 0, 1


def train(X, y, C_, gamma, tol, *, kind=RBF, max_iter=None, cache_bytes=8 << 30, threads=None,
          trace_len=0, want_f=False, selection=MVP) -> TrainResult:
    """Binary SMO (paper, Section III.B): maximal-violating-pair selection, or with
    ``selection=SECOND_ORDER`` the second-order rule for the second index of the pair."""
    lib = _load()
    X = _f32(X)
    y = np.ascontiguousarray(y, dtype=np.int32)
    n, d = X.shape
    if max_iter is None:
        max_iter = max(10_000_000, 100 * n)
    threads = max_threads() if threads is None else int(threads)
    alpha = np.zeros(n, dtype=np.float64)
    f = np.zeros(n, dtype=np.float64) if want_f else None
    res = _Res()
    tl = int(trace_len)
    tul = np.full((max(tl, 1), 2), -1, dtype=np.int32)
    tb = np.full((max(tl, 1), 2), np.nan, dtype=np.float64)
    tg = np.full((max(tl, 1), 2), np.nan, dtype=np.float64)
    rc = lib.oracle_train(_p(X), _p(y), n, d, int(kind), float(C_), float(gamma), float(tol), int(max_iter),
                          int(cache_bytes), threads, _p(alpha), _p(f) if f is not None else None, C.byref(res), tl,
                          _p(tul), _p(tb), _p(tg), int(selection))
    if rc < 0:
        raise ValueError(f"oracle_train rejected its input (status {rc})")
    steps = min(tl, int(res.iterations) + 1) if tl else 0
    return TrainResult(alpha=alpha, b=res.b, b_up=res.b_up, b_low=res.b_low, dual_obj=res.dual_obj,
                       iterations=int(res.iterations), n_sv=int(res.n_sv), n_bound=int(res.n_bound),
                       status=int(res.status), f=f,
                       trace_ul=tul[:steps].copy() if tl else None, trace_b=tb[:steps].copy() if tl else None,
                       trace_gap=tg[:steps].copy() if tl else None)


# Working-set variant: local tolerance factor and per-round step cap used unless given.
WS_FRAC = 0.5
WS_INNER_PER_Q = 100


@dataclass
class WsResult(TrainResult):
    rounds: int = 0
    ws_trace: np.ndarray | None = None      # [rounds, q] int32 working sets, -1 padded
    trace_margin: np.ndarray | None = None  # [rounds] smallest distance of a decision from flipping
    trace_t: np.ndarray | None = None       # [rounds] steps taken before the round


def train_ws(X, y, C_, gamma, tol, q, *, kind=RBF, frac=WS_FRAC, max_inner=None, max_iter=None,
             cache_bytes=8 << 30, threads=None, trace_len=0, ws_trace_len=0, want_f=False) -> WsResult:
    """Working-set decomposition: rounds of two-multiplier SMO steps on q samples (q = 2 is
    the maximal-violating-pair SMO of ``train``)."""
    lib = _load()
    X = _f32(X)
    y = np.ascontiguousarray(y, dtype=np.int32)
    n, d = X.shape
    if max_iter is None:
        max_iter = max(10_000_000, 100 * n)
    if max_inner is None:
        max_inner = WS_INNER_PER_Q * int(q)
    threads = max_threads() if threads is None else int(threads)
    alpha = np.zeros(n, dtype=np.float64)
    f = np.zeros(n, dtype=np.float64) if want_f else None
    res = _Res()
    rounds = C.c_int64(0)
    tl, wl = int(trace_len), int(ws_trace_len)
    tul = np.full((max(tl, 1), 2), -1, dtype=np.int32)
    tb = np.full((max(tl, 1), 2), np.nan, dtype=np.float64)
    tm = np.full(max(tl, 1), np.nan, dtype=np.float64)
    tt = np.full(max(tl, 1), -1, dtype=np.int64)
    wst = np.full((max(wl, 1), int(q)), -1, dtype=np.int32)
    rc = lib.oracle_train_ws(_p(X), _p(y), n, d, int(kind), float(C_), float(gamma), float(tol), int(q), float(frac),
                             int(max_inner), int(max_iter), int(cache_bytes), threads, _p(alpha),
                             _p(f) if f is not None else None, C.byref(res), C.byref(rounds), tl, _p(tul), _p(tb),
                             _p(tm), _p(tt), wl, _p(wst))
    if rc < 0:
        raise ValueError(f"oracle_train_ws rejected its input (status {rc})")
    r = int(rounds.value)
    steps = min(tl, r + 1) if tl else 0
    return WsResult(alpha=alpha, b=res.b, b_up=res.b_up, b_low=res.b_low, dual_obj=res.dual_obj,
                    iterations=int(res.iterations), n_sv=int(res.n_sv), n_bound=int(res.n_bound),
                    status=int(res.status), f=f,
                    trace_ul=tul[:steps].copy() if tl else None, trace_b=tb[:steps].copy() if tl else None,
                    rounds=r, ws_trace=wst[:min(wl, r)].copy() if wl else None,
                    trace_margin=tm[:steps].copy() if tl else None, trace_t=tt[:steps].copy() if tl else None)


def ws_select(f, y, alpha, C_, q) -> np.ndarray:
    """The working set a round of ``train_ws`` takes for the given f and alpha."""
    f = np.ascontiguousarray(f, dtype=np.float64)
    y = np.ascontiguousarray(y, dtype=np.int32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    B = np.full(int(q), -1, dtype=np.int64)
    m = _load().oracle_ws_select(_p(f), _p(y), _p(alpha), f.shape[0], float(C_), int(q), _p(B))
    if m < 0:
        raise ValueError("oracle_ws_select rejected its input")
    return B[:m].copy()


def kernel_value(a, b, gamma, kind=RBF) -> float:
    a = _f32(a).ravel()
    b = _f32(b).ravel()
    return float(_load().oracle_kernel_value(_p(a), _p(b), a.shape[0], int(kind), float(gamma)))


def kernel_rows(X, rows, gamma, kind=RBF, threads=None) -> np.ndarray:
    """K(x_r, x_j) for each requested r and every j (fp64)."""
    X = _f32(X)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    n, d = X.shape
    out = np.empty((rows.shape[0], n), dtype=np.float64)
    _load().oracle_kernel_rows(_p(X), n, d, _p(rows), rows.shape[0], int(kind), float(gamma), _p(out),
                               max_threads() if threads is None else int(threads))
    return out


def decision(X, y, alpha, b, T, gamma, kind=RBF, threads=None) -> np.ndarray:
    """d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b for every row x of T."""
    X = _f32(X)
    T = _f32(T)
    y = np.ascontiguousarray(y, dtype=np.int32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    n, d = X.shape
    m = T.shape[0]
    out = np.empty(m, dtype=np.float64)
    _load().oracle_decision(_p(X), _p(y), _p(alpha), float(b), n, d, int(kind), float(gamma), _p(T), m, _p(out),
                            max_threads() if threads is None else int(threads))
    return out


def f_from_alpha(X, y, alpha, gamma, rows=None, kind=RBF, threads=None) -> np.ndarray:
    """f_i = sum_j a_j y_j K_ij - y_i recomputed from alpha (listed rows, default all)."""
    X = _f32(X)
    y = np.ascontiguousarray(y, dtype=np.int32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    n, d = X.shape
    rows = np.arange(n, dtype=np.int64) if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty(rows.shape[0], dtype=np.float64)
    _load().oracle_f_from_alpha(_p(X), _p(y), _p(alpha), n, d, int(kind), float(gamma), _p(rows), rows.shape[0],
                                _p(out), max_threads() if threads is None else int(threads))
    return out


def ovo_pairs(k: int):
    return [(a, b) for a in range(k) for b in range(a + 1, k)]


def ovo_local(labels, a, b):
    """Local sample order of pair (a, b): class a by original index, then class b."""
    labels = np.asarray(labels)
    ia = np.flatnonzero(labels == a)
    ib = np.flatnonzero(labels == b)
    idx = np.concatenate([ia, ib])
    y = np.concatenate([np.ones(ia.shape[0], np.int32), -np.ones(ib.shape[0], np.int32)])
    return idx, y


def train_ovo(X, labels, k, C_, gamma, tol, **kw):
    """One-vs-one: one binary SMO per pair (a<b), class a = +1."""
    out = []
    for a, b in ovo_pairs(k):
        idx, y = ovo_local(labels, a, b)
        out.append((idx, y, train(X[idx], y, C_, gamma, tol, **kw)))
    return out


def predict_ovo(X, labels, k, models, T, gamma, threads=None):
    """Decision values [m, P] and voted class per test point."""
    T = _f32(T)
    m = T.shape[0]
    pairs = ovo_pairs(k)
    dec = np.empty((m, len(pairs)), dtype=np.float64)
    votes = np.zeros((m, k), dtype=np.int64)
    for p, ((a, b), (idx, y, r)) in enumerate(zip(pairs, models)):
        dec[:, p] = decision(X[idx], y, r.alpha, r.b, T, gamma, threads=threads)
        win = np.where(dec[:, p] > 0, a, b)
        votes[np.arange(m), win] += 1
    pred = np.argmax(votes, axis=1).astype(np.int32)  # argmax returns the first (smallest) class on ties
    return dec, pred
