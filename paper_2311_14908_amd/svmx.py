"""Python binding of libsvmx.so: the C entry points of include/svmx.h under the same names.

Argument marshalling only.  Device buffers are torch tensors on the current HIP device,
workspaces are ``torch.empty(bytes, dtype=torch.uint8)`` of the size the library asks for,
and work runs on ``torch.cuda.current_stream()``.  Every computation happens in the HIP
library; if it is not built this module raises on import of the library (there is no
fallback path).
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np
import torch

from .build import lib_path

SVM_OK, SVM_NOT_CONVERGED = 0, 1
SVM_EINVAL, SVM_ENOMEM, SVM_EDEVICE, SVM_EWORKSPACE = -1, -2, -3, -4
GRAM_AUTO, GRAM_ON, GRAM_OFF = 0, 1, 2
MFMA_SPLIT_F16, MFMA_F32 = 0, 1
SELECT_MVP, SELECT_SECOND_ORDER = 0, 1
WORKING_SET_AUTO = -1


class SvmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"svmx status {status}: {msg}")
        self.status = status


class svm_options(C.Structure):
    _fields_ = [("struct_size", C.c_int32), ("gram", C.c_int32), ("gram_budget_bytes", C.c_int64),
                ("row_cache_bytes", C.c_int64), ("max_iter", C.c_int64), ("check_every", C.c_int32),
                ("trace_len", C.c_int32), ("trace_ws", C.POINTER(C.c_int32)), ("trace_b", C.POINTER(C.c_double)),
                ("f_out", C.c_void_p), ("stream", C.c_void_p), ("workgroups", C.c_int32),
                ("exchange_levels", C.c_int32), ("gram_mfma", C.c_int32), ("working_set", C.c_int32),
                ("resident_rows", C.c_int32), ("selection", C.c_int32), ("reserved", C.c_int32),
                ("alpha_init", C.c_void_p), ("f_init", C.c_void_p)]


class svm_stats(C.Structure):
    _fields_ = [("iterations", C.c_int64), ("n_sv", C.c_int64), ("n_bound_sv", C.c_int64), ("b_up", C.c_double),
                ("b_low", C.c_double), ("dual_obj", C.c_double), ("gram_used", C.c_int32), ("launches", C.c_int32),
                ("t_gram", C.c_double), ("t_solve", C.c_double), ("t_finalize", C.c_double), ("t_total", C.c_double),
                ("t_kernel", C.c_double), ("rounds", C.c_int64),
                ("resident_rows", C.c_int32), ("schedule", C.c_int32), ("t_upload", C.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


EXPORTS = ("svm_default_options", "svm_train_workspace_bytes", "svm_train", "svm_train_static",
           "svm_predict_workspace_bytes",
           "svm_predict", "svm_train_ovo_workspace_bytes", "svm_train_ovo", "svm_predict_ovo_workspace_bytes",
           "svm_predict_ovo", "svm_kernel_rows", "svm_gram_workspace_bytes", "svm_gram", "svm_last_error")

_lib = None


def load(path: str | None = None):
    """Load libsvmx.so (raises if it has not been built)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or lib_path()
    if not os.path.exists(p):
        raise RuntimeError(f"{p} is missing: build it with paper_2311_14908_amd.build.build()")
    lib = C.CDLL(p)
    V, I64, I32, D = C.c_void_p, C.c_int64, C.c_int32, C.c_double
    OP, ST = C.POINTER(svm_options), C.POINTER(svm_stats)
    sig = {
        "svm_default_options": (None, [OP]),
        "svm_train_workspace_bytes": (I64, [I64, I64, OP]),
        "svm_train": (C.c_int, [V, V, I64, I64, D, D, D, V, C.POINTER(D), V, I64, OP, ST]),
        "svm_train_static": (C.c_int, [V, V, I64, I64, D, D, D, V, C.POINTER(D), OP, ST]),
        "svm_predict_workspace_bytes": (I64, [I64, I64, I64]),
        "svm_predict": (C.c_int, [V, V, V, D, I64, I64, D, V, I64, V, V, I64, OP]),
        "svm_train_ovo_workspace_bytes": (I64, [I64, I64, I32, OP]),
        "svm_train_ovo": (C.c_int, [V, V, I64, I64, I32, D, D, D, V, V, V, I64, OP, ST]),
        "svm_predict_ovo_workspace_bytes": (I64, [I64, I64, I32, I64]),
        "svm_predict_ovo": (C.c_int, [V, V, I64, I64, I32, V, V, D, V, I64, V, V, V, I64, OP]),
        "svm_kernel_rows": (C.c_int, [V, I64, I64, D, V, I64, V, OP]),
        "svm_gram_workspace_bytes": (I64, [I64, I64, OP]),
        "svm_gram": (C.c_int, [V, I64, I64, D, V, I64, V, I64, OP]),
        "svm_last_error": (C.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path is None:
        _lib = lib
    return lib


def _check(status: int, ok=(SVM_OK,)):
    if status not in ok:
        raise SvmError(status, load().svm_last_error().decode())
    return status


def _ptr(t: torch.Tensor | None):
    return None if t is None else C.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, dtype, name):
    if not (isinstance(t, torch.Tensor) and t.is_cuda):
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} tensor")
    return t


def options(gram=GRAM_AUTO, gram_budget_bytes=0, row_cache_bytes=0, max_iter=0, check_every=0, trace_len=0,
            workgroups=0, exchange_levels=0, gram_mfma=0, working_set=0, resident_rows=0, selection=0,
            f_out: torch.Tensor | None = None, stream=None, alpha_init: torch.Tensor | None = None,
            f_init: torch.Tensor | None = None):
    o = svm_options()
    load().svm_default_options(C.byref(o))
    o.gram = gram
    o.gram_budget_bytes = gram_budget_bytes
    o.row_cache_bytes = row_cache_bytes
    o.max_iter = max_iter
    if check_every:
        o.check_every = check_every
    o.trace_len = trace_len
    o.workgroups = workgroups
    o.exchange_levels = exchange_levels
    o.gram_mfma = gram_mfma
    o.working_set = working_set
    o.resident_rows = resident_rows
    o.selection = selection
    o.f_out = None if f_out is None else f_out.data_ptr()
    o.alpha_init = None if alpha_init is None else _dev(alpha_init, torch.float64, "alpha_init").data_ptr()
    o.f_init = None if f_init is None else _dev(f_init, torch.float64, "f_init").data_ptr()
    s = stream if stream is not None else torch.cuda.current_stream()
    o.stream = s.cuda_stream
    return o


@dataclass
class TrainOut:
    alpha: torch.Tensor
    b: float
    status: int
    stats: dict
    trace_ul: np.ndarray | None = None
    trace_b: np.ndarray | None = None


def svm_train(X: torch.Tensor, y: torch.Tensor, C_: float, gamma: float, tol: float, **opt) -> TrainOut:
    """Binary training; X fp32 [n,d], y int32 [n] in {+1,-1}, both on the device."""
    lib = load()
    _dev(X, torch.float32, "X")
    _dev(y, torch.int32, "y")
    n, d = X.shape
    o = options(**opt)
    tl = int(o.trace_len)
    tws = np.full(2 * max(tl, 1), -1, dtype=np.int32)
    tb = np.full(2 * max(tl, 1), np.nan, dtype=np.float64)
    if tl:
        o.trace_ws = tws.ctypes.data_as(C.POINTER(C.c_int32))
        o.trace_b = tb.ctypes.data_as(C.POINTER(C.c_double))
    wsb = lib.svm_train_workspace_bytes(n, d, C.byref(o))
    if wsb < 0:
        raise SvmError(SVM_EINVAL, "workspace size query failed")
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=X.device)
    alpha = torch.empty(n, dtype=torch.float64, device=X.device)
    b = C.c_double(0.0)
    st = svm_stats()
    status = _check(lib.svm_train(_ptr(X), _ptr(y), n, d, float(C_), float(gamma), float(tol), _ptr(alpha), C.byref(b),
                                  _ptr(ws), wsb, C.byref(o), C.byref(st)), ok=(SVM_OK, SVM_NOT_CONVERGED))
    out = TrainOut(alpha=alpha, b=b.value, status=status, stats=st.as_dict())
    if tl:
        steps = min(tl, (st.rounds if o.working_set > 0 else st.iterations) + 1)
        out.trace_ul = tws[:2 * steps].reshape(steps, 2).copy()
        out.trace_b = tb[:2 * steps].reshape(steps, 2).copy()
    return out


STATIC_SCRATCH_BYTES = 64 * 1024 * 1024


def svm_train_static(X: torch.Tensor, y: torch.Tensor, C_: float, gamma: float, tol: float, *,
                     alpha: torch.Tensor | None = None, **opt) -> TrainOut:
    """svm_train on the library's static device scratch (no workspace).  ``alpha`` may be given
    (a device fp64 [n] tensor) so that the call itself allocates nothing."""
    lib = load()
    _dev(X, torch.float32, "X")
    _dev(y, torch.int32, "y")
    n, d = X.shape
    o = options(**opt)
    tl = int(o.trace_len)
    tws = np.full(2 * max(tl, 1), -1, dtype=np.int32)
    tb = np.full(2 * max(tl, 1), np.nan, dtype=np.float64)
    if tl:
        o.trace_ws = tws.ctypes.data_as(C.POINTER(C.c_int32))
        o.trace_b = tb.ctypes.data_as(C.POINTER(C.c_double))
    if alpha is None:
        alpha = torch.empty(n, dtype=torch.float64, device=X.device)
    _dev(alpha, torch.float64, "alpha")
    b = C.c_double(0.0)
    st = svm_stats()
    status = _check(lib.svm_train_static(_ptr(X), _ptr(y), n, d, float(C_), float(gamma), float(tol), _ptr(alpha),
                                         C.byref(b), C.byref(o), C.byref(st)), ok=(SVM_OK, SVM_NOT_CONVERGED))
    out = TrainOut(alpha=alpha, b=b.value, status=status, stats=st.as_dict())
    if tl:
        steps = min(tl, (st.rounds if o.working_set > 0 else st.iterations) + 1)
        out.trace_ul = tws[:2 * steps].reshape(steps, 2).copy()
        out.trace_b = tb[:2 * steps].reshape(steps, 2).copy()
    return out


def svm_predict(X_train, y, alpha, b: float, gamma: float, X_test, **opt) -> torch.Tensor:
    lib = load()
    _dev(X_train, torch.float32, "X_train")
    _dev(y, torch.int32, "y")
    _dev(alpha, torch.float64, "alpha")
    _dev(X_test, torch.float32, "X_test")
    n, d = X_train.shape
    m = X_test.shape[0]
    o = options(**opt)
    wsb = lib.svm_predict_workspace_bytes(n, d, m)
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=X_train.device)
    dec = torch.empty(m, dtype=torch.float64, device=X_train.device)
    _check(lib.svm_predict(_ptr(X_train), _ptr(y), _ptr(alpha), float(b), n, d, float(gamma), _ptr(X_test), m,
                           _ptr(dec), _ptr(ws), wsb, C.byref(o)))
    return dec


@dataclass
class OvoOut:
    alpha: torch.Tensor  # packed [(k-1)*n]
    b: np.ndarray        # [P]
    status: int
    stats: list


def svm_train_ovo(X, label, k: int, C_: float, gamma: float, tol: float, **opt) -> OvoOut:
    lib = load()
    _dev(X, torch.float32, "X")
    _dev(label, torch.int32, "label")
    n, d = X.shape
    P = k * (k - 1) // 2
    o = options(**opt)
    wsb = lib.svm_train_ovo_workspace_bytes(n, d, k, C.byref(o))
    if wsb < 0:
        raise SvmError(SVM_EINVAL, "workspace size query failed")
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=X.device)
    alpha = torch.empty((k - 1) * n, dtype=torch.float64, device=X.device)
    b = np.zeros(P, dtype=np.float64)
    st = (svm_stats * P)()
    status = _check(lib.svm_train_ovo(_ptr(X), _ptr(label), n, d, int(k), float(C_), float(gamma), float(tol),
                                      _ptr(alpha), b.ctypes.data_as(C.c_void_p), _ptr(ws), wsb, C.byref(o), st),
                    ok=(SVM_OK, SVM_NOT_CONVERGED))
    return OvoOut(alpha=alpha, b=b, status=status, stats=[s.as_dict() for s in st])


def svm_predict_ovo(X, label, k: int, alpha, b: np.ndarray, gamma: float, X_test, **opt):
    lib = load()
    _dev(X, torch.float32, "X")
    _dev(label, torch.int32, "label")
    _dev(alpha, torch.float64, "alpha")
    _dev(X_test, torch.float32, "X_test")
    n, d = X.shape
    m = X_test.shape[0]
    P = k * (k - 1) // 2
    b = np.ascontiguousarray(b, dtype=np.float64)
    o = options(**opt)
    wsb = lib.svm_predict_ovo_workspace_bytes(n, d, k, m)
    ws = torch.empty(max(int(wsb), 1), dtype=torch.uint8, device=X.device)
    dec = torch.empty((m, P), dtype=torch.float64, device=X.device)
    pred = torch.empty(m, dtype=torch.int32, device=X.device)
    _check(lib.svm_predict_ovo(_ptr(X), _ptr(label), n, d, int(k), _ptr(alpha), b.ctypes.data_as(C.c_void_p),
                               float(gamma), _ptr(X_test), m, _ptr(dec), _ptr(pred), _ptr(ws), wsb, C.byref(o)))
    return dec, pred


def svm_kernel_rows(X, gamma: float, rows, **opt) -> torch.Tensor:
    lib = load()
    _dev(X, torch.float32, "X")
    n, d = X.shape
    rows_t = torch.as_tensor(rows, dtype=torch.int64).to(X.device).contiguous()
    out = torch.empty((rows_t.numel(), n), dtype=torch.float32, device=X.device)
    o = options(**opt)
    _check(lib.svm_kernel_rows(_ptr(X), n, d, float(gamma), _ptr(rows_t), rows_t.numel(), _ptr(out), C.byref(o)))
    return out


def svm_gram(X, gamma: float, ld: int | None = None, **opt) -> torch.Tensor:
    lib = load()
    _dev(X, torch.float32, "X")
    n, d = X.shape
    ld = n if ld is None else int(ld)
    G = torch.empty((n, ld), dtype=torch.float32, device=X.device)
    o = options(**opt)
    wsb = lib.svm_gram_workspace_bytes(n, d, C.byref(o))
    if wsb < 0:
        raise SvmError(SVM_EINVAL, "invalid sizes or options")
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=X.device)
    _check(lib.svm_gram(_ptr(X), n, d, float(gamma), _ptr(G), ld, _ptr(ws), wsb, C.byref(o)))
    return G



def svm_train_host(X: np.ndarray, y: np.ndarray, C_: float, gamma: float, tol: float, **opt):
    """Host-array convenience around svm_train: X (float32 [n, d]) and y (int32 [n]) are copied
    to the current device, trained there by the same call, and alpha comes back as a NumPy fp64
    array.  Returns (alpha, b, status, stats); the copies are the only difference."""
    Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
    yd = torch.from_numpy(np.ascontiguousarray(y, dtype=np.int32)).cuda()
    out = svm_train(Xd, yd, C_, gamma, tol, **opt)
    return out.alpha.cpu().numpy(), out.b, out.status, out.stats


def svm_predict_host(X_train: np.ndarray, y: np.ndarray, alpha: np.ndarray, b: float, gamma: float,
                     X_test: np.ndarray, **opt) -> np.ndarray:
    """Host-array convenience around svm_predict: the arrays are copied to the current device,
    the decision values (fp64 [m]) come back as a NumPy array."""
    dev = lambda a, t: torch.from_numpy(np.ascontiguousarray(a, dtype=t)).cuda()
    return svm_predict(dev(X_train, np.float32), dev(y, np.int32), dev(alpha, np.float64), b, gamma,
                       dev(X_test, np.float32), **opt).cpu().numpy()


def svm_train_ovo_host(X: np.ndarray, label: np.ndarray, k: int, C_: float, gamma: float, tol: float, **opt):
    """Host-array convenience around svm_train_ovo: returns (packed alpha as NumPy fp64, b [P],
    status, per-pair stats)."""
    Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.float32)).cuda()
    ld = torch.from_numpy(np.ascontiguousarray(label, dtype=np.int32)).cuda()
    out = svm_train_ovo(Xd, ld, k, C_, gamma, tol, **opt)
    return out.alpha.cpu().numpy(), out.b, out.status, out.stats


def svm_predict_ovo_host(X: np.ndarray, label: np.ndarray, k: int, alpha: np.ndarray, b: np.ndarray, gamma: float,
                         X_test: np.ndarray, **opt):
    """Host-array convenience around svm_predict_ovo: returns (decision values [m, P], predicted
    classes [m]) as NumPy arrays."""
    dev = lambda a, t: torch.from_numpy(np.ascontiguousarray(a, dtype=t)).cuda()
    dec, pred = svm_predict_ovo(dev(X, np.float32), dev(label, np.int32), k, dev(alpha, np.float64), b, gamma,
                                dev(X_test, np.float32), **opt)
    return dec.cpu().numpy(), pred.cpu().numpy()

def ovo_offsets(label: np.ndarray, k: int):
    """Start of each pair's block in the packed alpha of svm_train_ovo, and its size."""
    cnt = np.bincount(np.asarray(label), minlength=k)
    offs, sizes, o = [], [], 0
    for a in range(k):
        for b in range(a + 1, k):
            offs.append(o)
            sizes.append(int(cnt[a] + cnt[b]))
            o += int(cnt[a] + cnt[b])
    return np.array(offs), np.array(sizes)
