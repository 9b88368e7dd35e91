"""Host-side checks of libsvmx.so (no GPU needed): exports, defaults, workspace planning and
argument validation, which all run before any device access."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2311_14908_amd import svmx

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "svmx.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(svm_[a-z_]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(svmx.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = svmx.load()
    for name in declared_functions():
        assert hasattr(lib, name), name
    # and as dynamic symbols of the shared object
    out = os.popen(f"nm -D --defined-only {svmx.lib_path()}").read()
    for name in declared_functions():
        assert re.search(rf"\bT {name}$", out, flags=re.M), name


def test_struct_layouts_match_header():
    lib = svmx.load()
    o = svmx.svm_options()
    lib.svm_default_options(C.byref(o))
    assert o.struct_size == C.sizeof(svmx.svm_options) == 120
    assert o.selection == svmx.SELECT_MVP and o.reserved == 0
    assert o.alpha_init is None and o.f_init is None  # no warm start by default
    assert o.check_every == 65536 and o.gram == svmx.GRAM_AUTO
    assert C.sizeof(svmx.svm_stats) == 120


def _opts(**kw):
    lib = svmx.load()
    o = svmx.svm_options()
    lib.svm_default_options(C.byref(o))
    for k, v in kw.items():
        setattr(o, k, v)
    return o


def test_workspace_sizes():
    lib = svmx.load()
    ws = lambda n, d, **kw: lib.svm_train_workspace_bytes(n, d, C.byref(_opts(**kw)))
    # full Gram of the 100k x 32 workload: 100000 * ld(100032) * 4 bytes, plus small state and,
    # for the default split-fp16 Gram, its scratch (two fp16 halves of X, scales, norms)
    w3 = ws(100_000, 32)
    split = 2 * 2 * 100_000 * 32 + 8 * 100_000
    assert 4 * 100_000 * 100_032 + split <= w3 < 4 * 100_000 * 100_032 + split + (8 << 20)
    w3f = ws(100_000, 32, gram_mfma=svmx.MFMA_F32)
    assert 4 * 100_000 * 100_032 <= w3f < 4 * 100_000 * 100_032 + (8 << 20)
    # row path: no Gram
    assert ws(100_000, 32, gram=svmx.GRAM_OFF) < (16 << 20)
    # a Gram budget below the Gram size selects the row path under AUTO
    assert ws(20_000, 784, gram_budget_bytes=1 << 20) < (8 << 20)
    assert ws(20_000, 784, gram=svmx.GRAM_ON, gram_budget_bytes=1 << 20) > 4 * 20_000 ** 2
    # row cache adds cap * ld floats
    base = ws(5000, 16, gram=svmx.GRAM_OFF)
    withc = ws(5000, 16, gram=svmx.GRAM_OFF, row_cache_bytes=100 * 4 * 5056)
    assert withc - base >= 100 * 4 * 5056
    assert ws(1, 16) == -1 and ws(10, 0) == -1
    assert lib.svm_train_ovo_workspace_bytes(60_000, 784, 10, C.byref(_opts())) > 4 * 60_000 ** 2
    assert lib.svm_train_ovo_workspace_bytes(60_000, 784, 1, C.byref(_opts())) == -1
    bad = _opts()
    bad.struct_size = 12
    assert lib.svm_train_workspace_bytes(100, 4, C.byref(bad)) == -1


FAKE = C.c_void_p(0x1000)  # never dereferenced: every case below fails validation first


@pytest.mark.parametrize("case,expect", [
    (dict(X=None), svmx.SVM_EINVAL),
    (dict(y=None), svmx.SVM_EINVAL),
    (dict(n=1), svmx.SVM_EINVAL),
    (dict(d=0), svmx.SVM_EINVAL),
    (dict(Cv=0.0), svmx.SVM_EINVAL),
    (dict(Cv=float("inf")), svmx.SVM_EINVAL),
    (dict(gamma=-1.0), svmx.SVM_EINVAL),
    (dict(tol=float("nan")), svmx.SVM_EINVAL),
    (dict(wsb=16), svmx.SVM_EWORKSPACE),
    (dict(ws=None), svmx.SVM_EWORKSPACE),
    (dict(n=1 << 40, d=1 << 30), svmx.SVM_ENOMEM),  # n beyond the 32-bit sample index
    (dict(n=1 << 30, d=1 << 34), svmx.SVM_EINVAL),  # n*d bytes overflow int64
])
def test_train_rejects(case, expect):
    lib = svmx.load()
    a = dict(X=FAKE, y=FAKE, n=100, d=4, Cv=1.0, gamma=0.5, tol=1e-3, alpha=FAKE, ws=FAKE, wsb=16)
    a.update(case)
    b = C.c_double(0)
    o = _opts()
    st = lib.svm_train(a["X"], a["y"], a["n"], a["d"], a["Cv"], a["gamma"], a["tol"], a["alpha"], C.byref(b),
                       a["ws"], a["wsb"], C.byref(o), None)
    assert st == expect
    assert lib.svm_last_error().decode() != ""


@pytest.mark.parametrize("opt", [
    dict(selection=2),                                         # no such rule
    dict(reserved=1),                                          # reserved field must be 0
    dict(selection=svmx.SELECT_SECOND_ORDER, working_set=32),  # the working-set rounds have their own rule
    dict(selection=svmx.SELECT_SECOND_ORDER, gram=svmx.GRAM_OFF),  # row l is needed before l is known
    dict(selection=svmx.SELECT_SECOND_ORDER, gram_budget_bytes=1 << 10),  # AUTO falls back to the row path
])
def test_selection_option_rejects(opt):
    """Second-order selection runs on the Gram path of the per-step solver only; anything else is
    SVM_EINVAL, returned before any device access."""
    lib = svmx.load()
    o = _opts(**opt)
    b = C.c_double(0)
    st = lib.svm_train(FAKE, FAKE, 100, 4, 1.0, 0.5, 1e-3, FAKE, C.byref(b), FAKE, 1 << 40, C.byref(o), None)
    assert st == svmx.SVM_EINVAL
    assert lib.svm_last_error().decode() != ""
    if "gram" in opt or "gram_budget_bytes" in opt:
        bp = np.zeros(3).ctypes.data_as(C.c_void_p)
        assert lib.svm_train_ovo(FAKE, FAKE, 100, 4, 3, 1.0, 0.5, 1e-3, FAKE, bp, FAKE, 1 << 40, C.byref(o),
                                 None) == svmx.SVM_EINVAL
    else:
        assert lib.svm_train_workspace_bytes(100, 4, C.byref(o)) == -1


def test_working_set_auto_option():
    """working_set = SVM_WORKING_SET_AUTO plans for the rounds where they may run (binary, n > 4096,
    several owners, no trace), else for the per-step solver; other negative values are invalid."""
    lib = svmx.load()
    ws = lambda n, d, **kw: lib.svm_train_workspace_bytes(n, d, C.byref(_opts(**kw)))
    auto = svmx.WORKING_SET_AUTO
    assert ws(100_000, 32, working_set=auto) == ws(100_000, 32, working_set=32)
    assert ws(20_000, 784, working_set=auto) == ws(20_000, 784, working_set=128)
    assert ws(3000, 8, working_set=auto) == ws(3000, 8)  # small: one workgroup, per-step
    assert ws(100_000, 32, working_set=auto, trace_len=10) == ws(100_000, 32, trace_len=10)
    assert ws(100_000, 32, working_set=auto, selection=svmx.SELECT_SECOND_ORDER) == \
        ws(100_000, 32, selection=svmx.SELECT_SECOND_ORDER)
    assert ws(100_000, 32, working_set=-2) == -1 and ws(100_000, 32, working_set=3) == -1


def test_ovo_rejects():
    lib = svmx.load()
    b = np.zeros(100)
    o = _opts()
    bp = b.ctypes.data_as(C.c_void_p)
    assert lib.svm_train_ovo(FAKE, FAKE, 100, 4, 1, 1.0, 0.5, 1e-3, FAKE, bp, FAKE, 1 << 30, C.byref(o), None) == -1
    assert lib.svm_train_ovo(FAKE, FAKE, 100, 4, 65, 1.0, 0.5, 1e-3, FAKE, bp, FAKE, 1 << 30, C.byref(o), None) == -1
    assert lib.svm_train_ovo(FAKE, FAKE, 100, 4, 3, 1.0, 0.5, 1e-3, FAKE, bp, FAKE, 8, C.byref(o), None) == -4
    assert lib.svm_predict_ovo(FAKE, FAKE, 100, 4, 3, FAKE, None, 0.5, FAKE, 10, FAKE, FAKE, FAKE, 1 << 20,
                               C.byref(o)) == -1


def test_predict_and_rows_reject():
    lib = svmx.load()
    o = _opts()
    assert lib.svm_predict(FAKE, FAKE, FAKE, 0.0, 0, 4, 0.5, FAKE, 10, FAKE, FAKE, 256, C.byref(o)) == -1
    assert lib.svm_predict(FAKE, FAKE, FAKE, 0.0, 10, 4, 0.0, FAKE, 10, FAKE, FAKE, 256, C.byref(o)) == -1
    assert lib.svm_predict(FAKE, FAKE, FAKE, float("nan"), 10, 4, 0.5, FAKE, 10, FAKE, FAKE, 256, C.byref(o)) == -1
    assert lib.svm_kernel_rows(FAKE, 10, 4, 0.5, None, 2, FAKE, C.byref(o)) == -1
    assert lib.svm_gram(FAKE, 10, 4, 0.5, FAKE, 9, FAKE, 1 << 20, C.byref(o)) == -1
    assert lib.svm_gram(FAKE, 10, 4, -0.5, FAKE, 10, FAKE, 1 << 20, C.byref(o)) == -1
    # the split-fp16 Gram needs scratch: 2 halves x n x (d rounded up to 32) x 2 B + scales and norms
    assert lib.svm_gram_workspace_bytes(10, 4, C.byref(o)) >= 2 * 2 * 10 * 32 + 8 * 10
    assert lib.svm_gram(FAKE, 10, 4, 0.5, FAKE, 10, None, 0, C.byref(o)) == -4
    f32 = _opts(gram_mfma=svmx.MFMA_F32)
    assert lib.svm_gram_workspace_bytes(10, 4, C.byref(f32)) == 0
    bad = _opts(gram_mfma=7)
    assert lib.svm_gram_workspace_bytes(10, 4, C.byref(bad)) == -1


def test_working_set_options():
    lib = svmx.load()
    ws = lambda n, d, **kw: lib.svm_train_workspace_bytes(n, d, C.byref(_opts(**kw)))
    for q in (1, 3, 130, -2):
        assert ws(1000, 16, working_set=q) == -1, q
    for q in (2, 64, 128):
        assert ws(1000, 16, working_set=q) > 4 * 1000 * 1024, q
    # the candidate lists of 254 workgroups of 79 samples and 16 groups (two parities, 384 words
    # per list pair) in place of the pair solver's records
    w = ws(20_000, 784, working_set=128)
    assert w - ws(20_000, 784) >= 8 * 2 * (254 + 16) * 384 - 8 * 2 * (40 + 1) * 16
    # Gram path: n up to 255 workgroups of 1024 samples
    assert ws(261_120, 4, working_set=64, gram=svmx.GRAM_ON) > 0
    assert ws(261_121, 4, working_set=64, gram=svmx.GRAM_ON) == -1
    # row path: q x samples per workgroup <= 16384, and the split rows of X in the workspace
    for q, nmax in ((128, 255 * 128), (64, 255 * 256), (16, 255 * 1024)):
        assert ws(nmax, 8, working_set=q, gram=svmx.GRAM_OFF) > 0, q
        assert ws(nmax + 1, 8, working_set=q, gram=svmx.GRAM_OFF) == -1, q
    split = 2 * 2 * 20_000 * 800 + 8 * 20_000
    assert ws(20_000, 784, working_set=64, gram=svmx.GRAM_OFF) >= split
    st = lib.svm_train(FAKE, FAKE, 100, 4, 1.0, 0.5, 1e-3, FAKE, C.byref(C.c_double()), FAKE, 16,
                       C.byref(_opts(working_set=64, gram=svmx.GRAM_OFF)), None)
    assert st == svmx.SVM_EWORKSPACE


def test_predict_workspace_sizes():
    lib = svmx.load()
    for n, m in [(1, 0), (10, 0), (20_000, 0), (20_000, 1), (20_000, 10_000), (100_000, 129)]:
        w = lib.svm_predict_workspace_bytes(n, 16, m)
        assert w >= 12 * n + 8
        assert lib.svm_predict_ovo_workspace_bytes(max(n, 2), 16, 3, m) >= w
    assert lib.svm_predict_workspace_bytes(0, 16, 5) == -1
    assert lib.svm_predict_workspace_bytes(10, 16, -1) == -1


def test_predict_m0_is_noop():
    lib = svmx.load()
    o = _opts()
    assert lib.svm_predict(FAKE, FAKE, FAKE, 0.0, 10, 4, 0.5, None, 0, None, FAKE, 256, C.byref(o)) == 0


def test_resident_rows_option():
    """resident_rows: -1 (none), 0 (as many as fit) or a positive cap; below -1 is rejected.
    It does not change the workspace (the rows live in LDS)."""
    lib = svmx.load()
    ws = lambda n, d, **kw: lib.svm_train_workspace_bytes(n, d, C.byref(_opts(**kw)))
    base = ws(20_000, 784, gram=svmx.GRAM_OFF)
    assert base > 0
    for r in (-1, 0, 1, 1000):
        assert ws(20_000, 784, gram=svmx.GRAM_OFF, resident_rows=r) == base, r
    assert ws(20_000, 784, gram=svmx.GRAM_OFF, resident_rows=-2) == -1


def test_predict_ovo_workspace_covers_the_pair_chunks():
    """One-vs-one prediction runs up to 64 pairs per launch: its workspace holds, per pair of a
    chunk, room for all n samples' support vectors (12 bytes each) and the partial sums."""
    lib = svmx.load()
    n, d, m = 60_000, 784, 10_000
    one = lib.svm_predict_workspace_bytes(n, d, m)
    for k, pairs in ((2, 1), (10, 45), (12, 64), (64, 64)):
        w = lib.svm_predict_ovo_workspace_bytes(n, d, k, m)
        assert w >= 4 * n + pairs * 12 * n, k
        assert w >= one, k
    assert lib.svm_predict_ovo_workspace_bytes(n, d, 64, m) == lib.svm_predict_ovo_workspace_bytes(n, d, 12, m)
