"""GPU parity of the working-set solver (svm_options.working_set = q) through the C ABI, against
the oracle's working-set decomposition (oracle.train_ws) on identical seeded inputs.

Gates (fp64 oracle vs the fp32 Gram of the GPU path), as for the pair solver:
  rounds          the maximal violating pair of every round identical and b_up/b_low within 1e-4,
                  up to the first round in which the oracle takes a decision within 1e-5 of
                  flipping (its trace_margin); past such a tie the two trajectories may differ
  f, alpha        within 1e-4 / 1e-5 at a round boundary inside that window
  dual objective  relative error <= 1e-4
  decisions       max abs error <= 1e-3; labels compared on every point (a label may differ only
                  where the oracle's decision lies within the measured error of zero)
With q = 2 a round is one pair step, so the working-set kernel must reproduce the pair solver
bit for bit.  The list merges are exact and the f update sums in a fixed grouping, so results
do not depend on the number of workgroups or on the host check cadence.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2311_14908_amd import svmx, synth
from tests.label_checks import check_binary_labels, kkt_and_gap

pytestmark = pytest.mark.gpu

F_ATOL = 1e-4
W_RTOL = 1e-4
DEC_ATOL = 1e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    svmx.load()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def check_decisions(d_gpu, d_ref):
    err = float(np.max(np.abs(d_gpu - d_ref)))
    assert err <= DEC_ATOL
    check_binary_labels(d_gpu, d_ref, err)


C0 = synth.workload(0)


@pytest.fixture(scope="module")
def c0():
    X, y, Xt, _ = synth.generate(0)
    return X, y, Xt


def test_ws_q2_is_the_pair_solver(c0):
    X, y, _ = c0
    Xd, yd = dev(X), dev(y)
    pair = svmx.svm_train(Xd, yd, C0.C, C0.gamma, C0.tol, gram=svmx.GRAM_ON, trace_len=1001)
    ws = svmx.svm_train(Xd, yd, C0.C, C0.gamma, C0.tol, working_set=2, trace_len=1001)
    assert ws.stats["iterations"] == ws.stats["rounds"] == pair.stats["iterations"]
    assert torch.equal(ws.alpha, pair.alpha) and ws.b == pair.b
    np.testing.assert_array_equal(ws.trace_ul, pair.trace_ul)
    np.testing.assert_array_equal(ws.trace_b, pair.trace_b)
    ref = oracle.train(X, y, C0.C, C0.gamma, C0.tol, trace_len=1001)
    k = min(1000, ref.iterations + 1)
    np.testing.assert_array_equal(ws.trace_ul[:k], ref.trace_ul[:k])


TIE = 1e-5  # decisions closer than this to flipping may go either way with fp32 kernel values


def agree_window(ref):
    """Rounds whose trace both solvers must share: a decision of round r shows in the trace of
    round r + 1, so up to and including the first round whose oracle margin is below TIE."""
    near = np.flatnonzero(ref.trace_margin < TIE)
    return min(len(ref.trace_ul), int(near[0]) + 1 if near.size else len(ref.trace_ul))


@pytest.mark.parametrize("q", [4, 16, 64, 128])
def test_ws_c0_against_oracle(c0, q):
    """The rounds up to the first near tie against the oracle (pairs, b_up/b_low, and the state
    at a round boundary inside that window), then the optimum and the decisions."""
    X, y, Xt = c0
    ref = oracle.train_ws(X, y, C0.C, C0.gamma, C0.tol, q, trace_len=2000, want_f=True)
    out = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, working_set=q, trace_len=2000)
    assert out.status == svmx.SVM_OK
    k = agree_window(ref)
    np.testing.assert_array_equal(out.trace_ul[:k], ref.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], ref.trace_b[:k], atol=F_ATOL, rtol=0)
    # state at the start of the window's last round: both solvers stop there on max_iter
    t_cut = int(ref.trace_t[k - 1])
    if t_cut > 0:
        cut = oracle.train_ws(X, y, C0.C, C0.gamma, C0.tol, q, max_iter=t_cut, want_f=True)
        f = torch.empty(X.shape[0], dtype=torch.float64, device="cuda")
        part = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, working_set=q, max_iter=t_cut, f_out=f)
        assert part.stats["rounds"] == cut.rounds == k - 1
        np.testing.assert_allclose(part.alpha.cpu().numpy(), cut.alpha, atol=1e-5, rtol=0)
        assert np.max(np.abs(f.cpu().numpy() - cut.f)) <= F_ATOL
    st = out.stats
    assert abs(st["dual_obj"] - ref.dual_obj) <= W_RTOL * abs(ref.dual_obj)
    assert abs(st["rounds"] - ref.rounds) <= max(3, ref.rounds // 5)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= C0.C) and abs(a @ y) <= 1e-9 * C0.C * len(y)
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, C0.gamma, dev(Xt)).cpu().numpy()
    check_decisions(d_gpu, oracle.decision(X, y, ref.alpha, ref.b, Xt, C0.gamma))


@pytest.mark.parametrize("n,q,wgs", [(3, 128, 0), (50, 128, 0), (300, 64, 1), (1001, 16, 5), (4000, 64, 0),
                                     (5000, 128, 17), (3000, 128, 20), (2990, 32, 20), (6001, 2, 0),
                                     (20000, 128, 0)])
def test_ws_sizes_and_levels(n, q, wgs):
    """One workgroup, one merge level (up to 16 workgroups) and two levels (above 16), ragged
    slices (150 and 149 samples: the f update's thread mapping for slices of 129..192 samples;
    at q = 128 the Gram rows of B over the first 128 samples of a slice come from LDS and the
    rest from HBM), working sets larger than the problem:
    the rounds up to the first near tie against
    the oracle, the optimum, feasibility and decisions.  tol = 1e-5: past a near tie the two
    solvers stop at different points of the tol-optimal set, whose decisions may differ by about
    tol, so the comparison of the optimum is made where that spread is far below the gate."""
    X, y = synth.two_blobs(n, 6, seed=n)
    if n == 3:
        y = np.array([1, -1, 1], np.int32)
    ref = oracle.train_ws(X, y, 1.0, 0.3, 1e-5, q, trace_len=400)
    out = svmx.svm_train(dev(X), dev(y), 1.0, 0.3, 1e-5, working_set=q, workgroups=wgs, trace_len=400)
    assert out.status == svmx.SVM_OK
    k = agree_window(ref)
    np.testing.assert_array_equal(out.trace_ul[:k], ref.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], ref.trace_b[:k], atol=F_ATOL, rtol=0)
    assert abs(out.stats["dual_obj"] - ref.dual_obj) <= W_RTOL * abs(ref.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= 1.0) and abs(a @ y) <= 1e-9 * len(y)
    T = X[: min(n, 500)]
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, 0.3, dev(T)).cpu().numpy()
    check_decisions(d_gpu, oracle.decision(X, y, ref.alpha, ref.b, T, 0.3))


@pytest.mark.parametrize("q", [64, 32])
def test_ws_configurations_agree(q):
    """Workgroup counts (one merge level and two) and host check cadences change nothing: with 9
    workgroups a slice holds 1,000 samples, so the f update reads the Gram rows of B over the
    first 16,384 / q of them (256 at q = 64, 512 at q = 32) from LDS and over the rest from HBM;
    with 64 or more every row comes from LDS."""
    X, y = synth.two_blobs(9000, 8, seed=17)
    Xd, yd = dev(X), dev(y)
    kw = dict(working_set=q, trace_len=500)
    base = svmx.svm_train(Xd, yd, 1.0, 0.3, 1e-3, workgroups=9, **kw)
    for wgs, ce in [(16, 0), (17, 0), (64, 0), (141, 0), (0, 0), (0, 1), (0, 500)]:
        out = svmx.svm_train(Xd, yd, 1.0, 0.3, 1e-3, workgroups=wgs, check_every=ce, **kw)
        assert out.stats["iterations"] == base.stats["iterations"], (wgs, ce)
        assert out.stats["rounds"] == base.stats["rounds"], (wgs, ce)
        np.testing.assert_array_equal(out.trace_ul, base.trace_ul)
        np.testing.assert_array_equal(out.trace_b, base.trace_b)
        assert torch.equal(out.alpha, base.alpha) and out.b == base.b, (wgs, ce)


def test_ws_max_iter_not_converged_feasible():
    X, y = synth.two_blobs(2000, 5, seed=4)
    ref = oracle.train_ws(X, y, 1.0, 0.2, 1e-6, 32, max_iter=37, want_f=True)
    f = torch.empty(2000, dtype=torch.float64, device="cuda")
    out = svmx.svm_train(dev(X), dev(y), 1.0, 0.2, 1e-6, working_set=32, max_iter=37, f_out=f)
    assert out.status == svmx.SVM_NOT_CONVERGED and ref.status == 1
    assert out.stats["iterations"] == ref.iterations == 37
    assert out.stats["rounds"] == ref.rounds
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= 1.0) and abs(a @ y) <= 1e-12 * len(y)
    np.testing.assert_allclose(a, ref.alpha, atol=1e-5, rtol=0)
    assert np.max(np.abs(f.cpu().numpy() - ref.f)) <= F_ATOL


# --- row path: every round evaluates K(B, .) from X ---------------------------------------

@pytest.mark.parametrize("q", [16, 64, 128])
def test_ws_row_path_c0_against_oracle(c0, q):
    X, y, Xt = c0
    ref = oracle.train_ws(X, y, C0.C, C0.gamma, C0.tol, q, trace_len=2000)
    out = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, working_set=q, gram=svmx.GRAM_OFF, trace_len=2000)
    assert out.status == svmx.SVM_OK and out.stats["gram_used"] == 0
    k = agree_window(ref)
    np.testing.assert_array_equal(out.trace_ul[:k], ref.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], ref.trace_b[:k], atol=F_ATOL, rtol=0)
    assert abs(out.stats["dual_obj"] - ref.dual_obj) <= W_RTOL * abs(ref.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= C0.C) and abs(a @ y) <= 1e-9 * C0.C * len(y)
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, C0.gamma, dev(Xt)).cpu().numpy()
    check_decisions(d_gpu, oracle.decision(X, y, ref.alpha, ref.b, Xt, C0.gamma))


@pytest.mark.parametrize("cid,n,d,q,wgs", [(0, 3, 6, 128, 0), (0, 50, 6, 128, 0), (0, 1001, 6, 16, 5),
                                           (0, 4000, 6, 64, 0), (0, 5000, 13, 128, 0), (1, 2000, 784, 64, 0),
                                           (2, 3001, 128, 32, 0)])
def test_ws_row_path_sizes(cid, n, d, q, wgs):
    """Two to 63 owners, one and two merge levels, ragged blocks of samples (the MFMA tiles of
    16 and the blocks of 128 columns), one to 25 feature chunks of 32: the rounds up to the
    first near tie against the oracle, the optimum, feasibility and decisions (tol 1e-5)."""
    wl = synth.workload(cid)
    if cid == 0:
        X, y = synth.two_blobs(n, d, seed=n + d)
        if n == 3:
            y = np.array([1, -1, 1], np.int32)
        C_, g = 1.0, 0.3
    else:
        X, y, _, _ = synth.generate(cid, n=n, m=1, d=d)
        C_, g = wl.C, wl.gamma
    ref = oracle.train_ws(X, y, C_, g, 1e-5, q, trace_len=400)
    out = svmx.svm_train(dev(X), dev(y), C_, g, 1e-5, working_set=q, workgroups=wgs, gram=svmx.GRAM_OFF, trace_len=400)
    assert out.status == svmx.SVM_OK
    k = agree_window(ref)
    np.testing.assert_array_equal(out.trace_ul[:k], ref.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], ref.trace_b[:k], atol=F_ATOL, rtol=0)
    assert abs(out.stats["dual_obj"] - ref.dual_obj) <= W_RTOL * abs(ref.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= C_) and abs(a @ y) <= 1e-9 * C_ * len(y)
    T = X[: min(n, 500)]
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, g, dev(T)).cpu().numpy()
    check_decisions(d_gpu, oracle.decision(X, y, ref.alpha, ref.b, T, g))


def test_ws_row_path_configurations_agree():
    """Every kernel value is computed from its two rows alone, so the owner count changes
    nothing: bitwise equal results for 2 to 79 owners and any check cadence."""
    X, y, _, _ = synth.generate(1, n=6000, m=1, d=200)
    Xd, yd = dev(X), dev(y)
    kw = dict(working_set=64, gram=svmx.GRAM_OFF, trace_len=300)
    base = svmx.svm_train(Xd, yd, 10.0, 0.05, 1e-3, workgroups=24, **kw)
    for wgs, ce in [(2, 0), (16, 0), (17, 0), (0, 0), (0, 300)]:
        out = svmx.svm_train(Xd, yd, 10.0, 0.05, 1e-3, workgroups=wgs, check_every=ce, **kw)
        assert out.stats["rounds"] == base.stats["rounds"], (wgs, ce)
        np.testing.assert_array_equal(out.trace_ul, base.trace_ul)
        assert torch.equal(out.alpha, base.alpha) and out.b == base.b, (wgs, ce)


@pytest.mark.parametrize("cid,n,gram", [(3, 30_000, svmx.GRAM_ON), (2, 30_000, svmx.GRAM_ON), (1, 8_000, svmx.GRAM_OFF),
                                        (3, 30_000, svmx.GRAM_OFF)])
def test_auto_is_the_schedule_it_reports(cid, n, gram):
    """working_set = AUTO: when the rule keeps the rounds, the result is that of the explicit
    working set, bit for bit; when it hands over to the pair solver, the probe took exactly 128
    rounds and the pair steps reach the same optimum as the pair solver alone (W, tol-KKT on every
    row with f recomputed by the oracle).  The choice and the result do not depend on the host
    check cadence."""
    wl = synth.workload(cid)
    X, y, _, _ = synth.generate(cid, n=n, m=1)
    Xd, yd = dev(X), dev(y)
    auto = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=svmx.WORKING_SET_AUTO)
    st = auto.stats
    q = (64 if gram != svmx.GRAM_OFF else 128) if X.shape[1] >= 256 else 32
    print(f"\nworkload {cid} n={n} gram={gram}: schedule {st['schedule']}, {st['rounds']} rounds, "
          f"{st['iterations']} pair steps")
    assert auto.status == svmx.SVM_OK and st["schedule"] in (1, 2)
    if st["schedule"] == 1:
        w = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=q)
        assert torch.equal(w.alpha, auto.alpha) and w.b == auto.b
        assert w.stats["rounds"] == st["rounds"] and w.stats["iterations"] == st["iterations"]
    else:
        assert st["rounds"] == 128
        pair = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram)
        assert abs(st["dual_obj"] - pair.stats["dual_obj"]) <= W_RTOL * abs(pair.stats["dual_obj"])
        a = auto.alpha.cpu().numpy()
        assert np.all(a >= 0) and np.all(a <= wl.C) and abs(float(a @ y)) <= 1e-9 * wl.C * len(y)
        f = oracle.f_from_alpha(X, y, a, wl.gamma)
        kkt_and_gap(f, y, a, auto.b, wl.C, wl.tol, slack=1e-4)
    other = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=svmx.WORKING_SET_AUTO,
                           check_every=333)
    assert other.stats["schedule"] == st["schedule"]
    assert torch.equal(other.alpha, auto.alpha) and other.b == auto.b
