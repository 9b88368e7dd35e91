"""Second-order selection on the GPU (option selection = SELECT_SECOND_ORDER, Gram path) against
the oracle's second-order solve (oracle.train(..., selection=oracle.SECOND_ORDER)), through the
C ABI.

The paper cites two working-pair rules for SMO (Section III.B).  With the second-order one, u is
the smallest f over I_up as before and l maximises (f_t - f_u)^2 / a_ut over the members t of
I_low above f_u.  Gates:
  working set   identical (u, l) up to the first step where the oracle's choice is within
                rounding of another (u: runner-up gap below 1e-6; l: best two gains within
                1e-4 relative -- a gain carries the fp32 kernel error of f and of K_ut)
  optimum       W within 1e-4 relative, decisions within 1e-3, labels on every point, tol-KKT
                and the duality gap on every row with f recomputed by the oracle
  exactness     bit-identical alpha and trace for any workgroup count and exchange depth, and
                one-vs-one pairs equal to standalone binary solves
The optimum does not depend on the selection rule (the RBF dual has a unique solution), so at
the full workload sizes the GPU's second-order solution is checked against the stored oracle
optimum of the first-order solve.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2311_14908_amd import svmx, synth
from tests.label_checks import check_binary_labels, kkt_and_gap

pytestmark = pytest.mark.gpu

SO = svmx.SELECT_SECOND_ORDER
GAP_U, GAP_L = 1e-6, 1e-4
W_RTOL, DEC_ATOL = 1e-4, 1e-3
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    svmx.load()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def comparable_steps(ref, limit):
    """Steps of the oracle's trace before its first near-tie (see the module docstring)."""
    g = np.asarray(ref.trace_gap)
    last = min(ref.iterations + 1, limit, g.shape[0])
    near = np.flatnonzero((g[1:last, 0] < GAP_U) | (g[1:last, 1] < GAP_L))
    return int(near[0]) + 1 if near.size else last


C0 = synth.workload(0)


@pytest.fixture(scope="module")
def c0so():
    X, y, Xt, _ = synth.generate(0)
    ref = oracle.train(X, y, C0.C, C0.gamma, C0.tol, trace_len=5000, selection=oracle.SECOND_ORDER)
    return X, y, Xt, ref


CONFIGS = [(0, 0, svmx.MFMA_SPLIT_F16), (3, 0, svmx.MFMA_SPLIT_F16), (8, 0, svmx.MFMA_SPLIT_F16),
           (8, 2, svmx.MFMA_SPLIT_F16), (0, 0, svmx.MFMA_F32)]


@pytest.mark.parametrize("wgs,levels,mfma", CONFIGS)
def test_c0_trace_and_optimum(c0so, wgs, levels, mfma):
    X, y, Xt, ref = c0so
    out = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, gram=svmx.GRAM_ON, workgroups=wgs,
                         exchange_levels=levels, gram_mfma=mfma, trace_len=1001, selection=SO)
    assert out.status == svmx.SVM_OK
    st = out.stats
    k = comparable_steps(ref, 1001)
    assert k >= 300
    same = np.all(out.trace_ul[:k] == ref.trace_ul[:k], axis=1)
    first = int(np.argmin(same)) if not same.all() else k
    print(f"\n{wgs} workgroups, {levels} levels: gpu {st['iterations']} steps, oracle {ref.iterations}; "
          f"traces equal for {first} of {k} comparable steps")
    np.testing.assert_array_equal(out.trace_ul[:k], ref.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], ref.trace_b[:k], atol=1e-4, rtol=0)
    assert abs(st["dual_obj"] - ref.dual_obj) <= W_RTOL * abs(ref.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= C0.C) and abs(a @ y) <= 1e-9 * C0.C * len(y)
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, C0.gamma, dev(Xt)).cpu().numpy()
    d_ref = oracle.decision(X, y, ref.alpha, ref.b, Xt, C0.gamma)
    err = float(np.max(np.abs(d_gpu - d_ref)))
    assert err <= DEC_ATOL
    check_binary_labels(d_gpu, d_ref, err)
    f = oracle.f_from_alpha(X, y, a, C0.gamma)
    kkt_and_gap(f, y, a, out.b, C0.C, C0.tol, slack=1e-4)


def test_exchange_is_exact_for_second_order():
    """Both exchanges of a step are exact reductions: 1, 5, 16 and 40 workgroups (one and two
    exchange levels) give the same alpha, b and trace, bit for bit."""
    X, y = synth.two_blobs(6000, 24, seed=31)
    runs = []
    for wgs, levels in [(1, 0), (5, 0), (16, 2), (40, 0), (40, 2)]:
        out = svmx.svm_train(dev(X), dev(y), 2.0, 1.0 / 24, 1e-3, gram=svmx.GRAM_ON, workgroups=wgs,
                             exchange_levels=levels, trace_len=3000, selection=SO)
        assert out.status == svmx.SVM_OK
        runs.append(out)
    for o in runs[1:]:
        assert o.stats["iterations"] == runs[0].stats["iterations"]
        assert torch.equal(o.alpha, runs[0].alpha) and o.b == runs[0].b
        np.testing.assert_array_equal(o.trace_ul, runs[0].trace_ul)


def test_second_order_independent_of_check_cadence():
    """A launch boundary between the two exchanges of a step's selection never happens: a launch
    ends at the start of a step.  Launches of 1, 7 and 256 steps give the same result."""
    X, y = synth.two_blobs(5000, 8, seed=4)
    ref = None
    for ce in (1, 7, 256, 0):
        out = svmx.svm_train(dev(X), dev(y), 1.0, 0.125, 1e-3, gram=svmx.GRAM_ON, check_every=ce, workgroups=6,
                             selection=SO, max_iter=900, trace_len=900)
        if ref is None:
            ref = out
            continue
        assert out.stats["iterations"] == ref.stats["iterations"]
        assert torch.equal(out.alpha, ref.alpha)
        np.testing.assert_array_equal(out.trace_ul, ref.trace_ul)


def test_ovo_pairs_equal_standalone_second_order_solves():
    k = 4
    X, lab, _, _ = synth.generate(4, n=800, m=1, d=24, classes=k)
    out = svmx.svm_train_ovo(dev(X), dev(lab), k, 10.0, 0.05, 1e-3, gram=svmx.GRAM_ON, selection=SO)
    offs, sizes = svmx.ovo_offsets(lab, k)
    for p, (a, b) in enumerate(oracle.ovo_pairs(k)):
        idx, y = oracle.ovo_local(lab, a, b)
        r = svmx.svm_train(dev(X[idx]), dev(y), 10.0, 0.05, 1e-3, gram=svmx.GRAM_ON, selection=SO)
        assert torch.equal(out.alpha[offs[p]:offs[p] + sizes[p]], r.alpha)
        assert out.b[p] == r.b
        assert out.stats[p]["iterations"] == r.stats["iterations"]


def test_second_order_takes_no_more_steps_than_mvp_on_c0(c0so):
    """On workload 0 the second-order rule needs fewer steps than the maximal violating pair, on
    both sides (oracle: 424 against 498)."""
    X, y, _, ref = c0so
    mvp = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, gram=svmx.GRAM_ON)
    so = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, gram=svmx.GRAM_ON, selection=SO)
    assert so.stats["iterations"] < mvp.stats["iterations"]
    assert abs(so.stats["iterations"] - ref.iterations) <= 0.05 * ref.iterations


@pytest.mark.parametrize("cid", [1, 2, 3])
def test_second_order_full_size(cid):
    """The full binary workloads: the first steps against a truncated oracle second-order solve
    (up to its first near-tie), then the stored oracle optimum (W, decisions, labels) and tol-KKT
    and the duality gap on every row with f recomputed by the oracle from the GPU's alpha."""
    path = os.path.join(GOLDEN, f"oracle_full_w{cid}.json")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    R = json.load(open(path))
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid)
    nt = len(R["test_decisions"])
    steps = 300
    ref = oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=steps, trace_len=steps, cache_bytes=1 << 30,
                       selection=oracle.SECOND_ORDER)
    Xd, yd = dev(X), dev(y)
    out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, trace_len=steps, selection=SO)
    assert out.status == svmx.SVM_OK and out.stats["gram_used"] == 1
    st = out.stats
    print(f"\nworkload {cid}: second order {st['iterations']} steps in {st['t_solve']:.3f} s, W={st['dual_obj']:.9f}; "
          f"oracle (first order) {R['iterations']} steps, W={R['dual_obj']:.9f}")
    k = comparable_steps(ref, steps)
    assert k >= 20
    np.testing.assert_array_equal(out.trace_ul[:k], ref.trace_ul[:k])
    assert abs(st["dual_obj"] - R["dual_obj"]) <= W_RTOL * abs(R["dual_obj"])
    d_gpu = svmx.svm_predict(Xd, yd, out.alpha, out.b, wl.gamma, dev(Xt[:nt])).cpu().numpy()
    d_ref = np.array(R["test_decisions"])
    err = float(np.max(np.abs(d_gpu - d_ref)))
    assert err <= DEC_ATOL
    check_binary_labels(d_gpu, d_ref, err)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= wl.C) and abs(float(a @ y)) <= 1e-9 * wl.C * len(y)
    f = oracle.f_from_alpha(X, y, a, wl.gamma)
    gap, _ = kkt_and_gap(f, y, a, out.b, wl.C, wl.tol, slack=1e-4)
    print(f"decisions within {err:.2e}; duality gap {gap:.3e}")
