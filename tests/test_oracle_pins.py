"""Pins of the CPU oracle against what the mathematics fixes (no GPU).

Each test checks the oracle against something other than itself: closed forms,
exact enumeration of the QP, invariants computed through an independent route
(SciPy distances), a duality-gap certificate and an external library (LIBSVM via
scikit-learn).
"""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
from paper_2311_14908_amd import synth
from tests import bruteforce_qp as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rbf(X, Z, gamma):
    return np.exp(-gamma * cdist(X.astype(np.float64), Z.astype(np.float64), "sqeuclidean"))


def dual_W(K, y, a):
    v = a * y
    return float(a.sum() - 0.5 * v @ K @ v)


# --- closed forms -------------------------------------------------------------------

@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLDEN, "two_point.json")))["cases"])
def test_two_point_closed_form(case):
    X = np.array([case["x1"], case["x2"]], dtype=np.float32)
    y = np.array([1, -1], dtype=np.int32)
    kind = oracle.LINEAR if case["kernel"] == "linear" else oracle.RBF
    r = oracle.train(X, y, case["C"], case["gamma"], 1e-9, kind=kind)
    assert r.status == 0
    assert r.iterations == case["steps"]
    np.testing.assert_allclose(r.alpha, [case["alpha"]] * 2, rtol=1e-7, atol=0)
    assert abs(r.b - case["b"]) <= 1e-9
    if kind == oracle.LINEAR:
        w = r.alpha[0] * (X[0].astype(np.float64) - X[1])
        assert abs(np.linalg.norm(w) - case["w_norm"]) <= 1e-9
        # geometric margin 2/|w| equals the distance between the two points
        assert abs(2.0 / np.linalg.norm(w) - np.linalg.norm(X[0].astype(np.float64) - X[1])) <= 1e-9
        # both points sit on the margin: y_i d(x_i) = 1
        d = oracle.decision(X, y, r.alpha, r.b, X, 0.0, kind=oracle.LINEAR)
        np.testing.assert_allclose(d * y, [1.0, 1.0], atol=1e-9)


def test_linear_two_point_random():
    rng = np.random.default_rng(5)
    for _ in range(20):
        X = rng.standard_normal((2, 6)).astype(np.float32)
        D2 = float(((X[0].astype(np.float64) - X[1]) ** 2).sum())
        r = oracle.train(X, np.array([1, -1], np.int32), 10.0 / D2 + 1.0, 0.0, 1e-9, kind=oracle.LINEAR)
        np.testing.assert_allclose(r.alpha, 2.0 / D2, rtol=1e-9)
        nx = (X.astype(np.float64) ** 2).sum(1)
        assert abs(r.b - (nx[0] - nx[1]) / D2) <= 1e-9 * max(1.0, abs(r.b))


def test_first_step_closed_form():
    """Step 1 from a = 0: f = -y ties everywhere, so u/l are the first +1/-1 samples
    and both multipliers move to min(C, 2/eta) with eta = 2 - 2 K_ul (RBF)."""
    for cid in (0, 1, 2, 3):
        wl = synth.workload(cid)
        X, y, _, _ = synth.generate(cid, n=300, m=1)
        r = oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=1, trace_len=2)
        u = int(np.flatnonzero(y == 1)[0])
        l = int(np.flatnonzero(y == -1)[0])
        assert tuple(r.trace_ul[0]) == (u, l)
        eta = 2.0 - 2.0 * rbf(X[u:u + 1], X[l:l + 1], wl.gamma)[0, 0]
        a1 = min(wl.C, 2.0 / eta)
        np.testing.assert_allclose([r.alpha[u], r.alpha[l]], [a1, a1], rtol=1e-12)
        assert np.count_nonzero(r.alpha) == 2


# --- exact QP by enumeration -----------------------------------------------------------

def _tiny_problem(seed, n):
    rng = np.random.default_rng(seed)
    d = int(rng.integers(2, 6))
    X = rng.standard_normal((n, d)).astype(np.float32)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int32)
    y[0], y[1] = 1, -1
    gamma = float(rng.uniform(0.1, 1.5))
    C = float(rng.choice([0.3, 1.0, 5.0, 100.0]))
    return X, y, gamma, C


@pytest.mark.parametrize("seed", range(60))
def test_bruteforce_qp(seed):
    n = 3 + seed % 6  # 3..8
    X, y, gamma, C = _tiny_problem(seed, n)
    K = rbf(X, X, gamma)
    Q = (y[:, None] * y[None, :]) * K
    a_star, b_star, acc, has_free = bf.solve(Q, y, C)
    r = oracle.train(X, y, C, gamma, 1e-11)
    assert r.status == 0
    np.testing.assert_allclose(r.alpha, a_star, atol=1e-6)
    W_star = dual_W(K, y, a_star)
    assert abs(r.dual_obj - W_star) <= 1e-9 * max(1.0, abs(W_star))
    if has_free:
        assert abs(r.b - b_star) <= 1e-6


@pytest.mark.parametrize("seed", [1000, 1001])
def test_bruteforce_qp_n10(seed):
    X, y, gamma, C = _tiny_problem(seed, 10)
    K = rbf(X, X, gamma)
    Q = (y[:, None] * y[None, :]) * K
    a_star, b_star, _, has_free = bf.solve(Q, y, C)
    r = oracle.train(X, y, C, gamma, 1e-11)
    np.testing.assert_allclose(r.alpha, a_star, atol=1e-6)
    assert abs(r.dual_obj - dual_W(K, y, a_star)) <= 1e-9 * max(1.0, abs(r.dual_obj))


def test_bruteforce_catches_planted_mistake():
    """The enumeration pin is sharp: a solution with a dropped cross term is rejected."""
    X, y, gamma, C = _tiny_problem(7, 6)
    K = rbf(X, X, gamma)
    Q = (y[:, None] * y[None, :]) * K
    a_star, _, _, _ = bf.solve(Q, y, C)
    Kbad = np.diag(np.diag(K))  # kernel with the cross terms dropped
    Qbad = (y[:, None] * y[None, :]) * Kbad
    a_bad, _, _, _ = bf.solve(Qbad, y, C)
    assert np.max(np.abs(a_bad - a_star)) > 1e-3


# --- invariants along the trajectory ---------------------------------------------------

def test_invariants_every_step():
    X, y = synth.two_blobs(160, 5, seed=3)
    C, gamma = 1.0, 0.2
    K = rbf(X, X, gamma)
    prev_W = -np.inf
    full = oracle.train(X, y, C, gamma, 1e-3)
    for t in range(1, full.iterations + 1):
        r = oracle.train(X, y, C, gamma, 1e-3, max_iter=t, want_f=True)
        a = r.alpha
        assert abs(float(a @ y)) <= 1e-10 * C * len(y)
        assert np.all(a >= 0.0) and np.all(a <= C)
        f_direct = K @ (a * y) - y
        np.testing.assert_allclose(r.f, f_direct, atol=1e-9)
        W = dual_W(K, y, a)
        assert W > prev_W
        prev_W = W
        # the stored objective matches the direct a^T Q a form
        assert abs(r.dual_obj - W) <= 1e-9 * max(1.0, abs(W))


def test_selection_is_maximal_violating_pair():
    X, y = synth.two_blobs(120, 4, seed=11)
    C, gamma = 0.7, 0.3
    K = rbf(X, X, gamma)
    full = oracle.train(X, y, C, gamma, 1e-3, trace_len=10_000)
    for t in [0, 1, 2, 5, 17, full.iterations // 2, full.iterations - 1]:
        r = oracle.train(X, y, C, gamma, 1e-3, max_iter=t)
        a = r.alpha
        f = K @ (a * y) - y
        up = ((y > 0) & (a < C)) | ((y < 0) & (a > 0))
        low = ((y > 0) & (a > 0)) | ((y < 0) & (a < C))
        iu = np.flatnonzero(up)[np.argmin(f[up])]
        il = np.flatnonzero(low)[np.argmax(f[low])]
        assert tuple(full.trace_ul[t]) == (iu, il)


# --- termination certificate -----------------------------------------------------------

@pytest.mark.parametrize("cid", [0, 2, 3])
def test_kkt_and_duality_gap(cid):
    wl = synth.workload(cid)
    X, y, _, _ = synth.generate(cid, n=600, m=1)
    r = oracle.train(X, y, wl.C, wl.gamma, wl.tol)
    assert r.status == 0
    K = rbf(X, X, wl.gamma)
    a = r.alpha
    f = K @ (a * y) - y
    up = ((y > 0) & (a < wl.C)) | ((y < 0) & (a > 0))
    low = ((y > 0) & (a > 0)) | ((y < 0) & (a < wl.C))
    assert np.all(f[up] >= r.b - wl.tol / 2 - 1e-9)
    assert np.all(f[low] <= r.b + wl.tol / 2 + 1e-9)
    W = dual_W(K, y, a)
    v = a * y
    d = K @ v - r.b
    P = 0.5 * v @ K @ v + wl.C * np.maximum(0.0, 1.0 - y * d).sum()
    # P - W = sum_i [C xi_i + a_i (y_i d_i - 1)]; at a tol-KKT point every term is at most
    # C*tol (free: C tol/2 + a tol/2; at a bound: C tol/2), so the gap is at most n*C*tol.
    assert P - W >= -1e-9
    assert (P - W) <= len(y) * wl.C * wl.tol


# --- external library (different algorithm, same optimum) ------------------------------

def test_sklearn_same_optimum_c0():
    from sklearn.svm import SVC
    wl = synth.workload(0)
    X, y, Xt, yt = synth.generate(0)
    r = oracle.train(X, y, wl.C, wl.gamma, wl.tol)
    sk = SVC(kernel="rbf", C=wl.C, gamma=wl.gamma, tol=wl.tol, shrinking=False).fit(X.astype(np.float64), y)
    a_sk = np.zeros(len(y))
    a_sk[sk.support_] = np.abs(sk.dual_coef_[0])
    K = rbf(X, X, wl.gamma)
    W_o, W_s = dual_W(K, y, r.alpha), dual_W(K, y, a_sk)
    assert abs(W_o - W_s) <= 1e-4 * abs(W_s)
    d_o = oracle.decision(X, y, r.alpha, r.b, Xt, wl.gamma)
    d_s = sk.decision_function(Xt.astype(np.float64))
    assert np.max(np.abs(d_o - d_s)) <= 2e-2
    sure = np.abs(d_s) > 2e-2
    assert np.array_equal(d_o[sure] > 0, d_s[sure] > 0)


def test_tolerance_slack_c0():
    """How much of the decision budget tol=1e-3 itself uses (oracle at 1e-3 vs 1e-6)."""
    wl = synth.workload(0)
    X, y, Xt, _ = synth.generate(0)
    r3 = oracle.train(X, y, wl.C, wl.gamma, 1e-3)
    r6 = oracle.train(X, y, wl.C, wl.gamma, 1e-6)
    d3 = oracle.decision(X, y, r3.alpha, r3.b, Xt, wl.gamma)
    d6 = oracle.decision(X, y, r6.alpha, r6.b, Xt, wl.gamma)
    assert np.max(np.abs(d3 - d6)) < 5e-3
    assert abs(r3.dual_obj - r6.dual_obj) <= 1e-4 * abs(r6.dual_obj)


# --- one-vs-one bookkeeping -------------------------------------------------------------

def test_ovo_count_and_votes():
    X, lab = synth.multiclass_blobs(300, 6, 4, seed=2)
    models = oracle.train_ovo(X, lab, 4, 1.0, 0.5, 1e-3)
    assert len(models) == 4 * 3 // 2
    for (a, b), (idx, y, _) in zip(oracle.ovo_pairs(4), models):
        assert np.all(lab[idx[y > 0]] == a) and np.all(lab[idx[y < 0]] == b)
        assert np.all(np.diff(idx[y > 0]) > 0) and np.all(np.diff(idx[y < 0]) > 0)
    dec, pred = oracle.predict_ovo(X, lab, 4, models, X, 0.5)
    assert dec.shape == (300, 6)
    assert np.mean(pred == lab) > 0.8


def test_rejects_bad_input():
    X = np.zeros((4, 2), np.float32)
    with pytest.raises(ValueError):
        oracle.train(X, np.array([1, 1, 1, 1], np.int32), 1.0, 1.0, 1e-3)
    with pytest.raises(ValueError):
        oracle.train(X, np.array([1, -1, 2, 1], np.int32), 1.0, 1.0, 1e-3)
    with pytest.raises(ValueError):
        oracle.train(X, np.array([1, -1, 1, 1], np.int32), -1.0, 1.0, 1e-3)


def test_row_cache_does_not_change_results():
    X, y = synth.two_blobs(300, 4, seed=9)
    a = oracle.train(X, y, 1.0, 0.25, 1e-3, trace_len=5000)
    b = oracle.train(X, y, 1.0, 0.25, 1e-3, trace_len=5000, cache_bytes=8 * 300 * 3)
    np.testing.assert_array_equal(a.alpha, b.alpha)
    np.testing.assert_array_equal(a.trace_ul, b.trace_ul)


def test_thread_count_does_not_change_results():
    X, y = synth.two_blobs(300, 4, seed=10)
    a = oracle.train(X, y, 1.0, 0.25, 1e-3, threads=1)
    b = oracle.train(X, y, 1.0, 0.25, 1e-3, threads=4)
    np.testing.assert_array_equal(a.alpha, b.alpha)


# --- working-set decomposition (rounds of pair steps on q samples) ----------------------

@pytest.mark.parametrize("cid", [0, 2])
def test_ws_q2_is_the_pair_step(cid):
    """With q = 2 a round is exactly one maximal-violating-pair step: same pairs, same
    multipliers to the bit, same bias."""
    wl = synth.workload(cid)
    X, y, _, _ = synth.generate(cid, n=600, m=1)
    a = oracle.train(X, y, wl.C, wl.gamma, wl.tol, trace_len=5000)
    b = oracle.train_ws(X, y, wl.C, wl.gamma, wl.tol, 2, trace_len=5000)
    assert a.iterations == b.iterations == b.rounds
    assert np.array_equal(a.trace_ul, b.trace_ul)
    assert np.array_equal(a.alpha, b.alpha)
    assert a.b == b.b


def _lex_select(f, y, alpha, C, q):
    """The working-set rule written with NumPy's stable lexsort."""
    up = ((y > 0) & (alpha < C)) | ((y < 0) & (alpha > 0))
    low = ((y > 0) & (alpha > 0)) | ((y < 0) & (alpha < C))
    idx = np.arange(f.shape[0])
    fu, fl = f + 0.0, -f + 0.0  # +0.0 folds -0 into +0, as the comparisons do
    su = idx[up][np.lexsort((idx[up], fu[up]))][: q // 2]
    sl = idx[low][np.lexsort((idx[low], fl[low]))][: q // 2]
    return np.array(list(su) + [i for i in sl if i not in set(su)], dtype=np.int64)


@pytest.mark.parametrize("seed", range(8))
def test_ws_select_rule(seed):
    """Working sets against the rule evaluated independently, on values with many ties,
    signed zeros and every membership case."""
    rng = np.random.default_rng(seed)
    n = int(rng.integers(5, 400))
    C = 2.0
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int32)
    alpha = rng.choice([0.0, C, 0.7], size=n)
    f = np.round(rng.standard_normal(n), 1)
    f[rng.random(n) < 0.1] = -0.0
    f[rng.random(n) < 0.1] = 0.0
    for q in (2, 4, 10, 64, 2 * n + 2):
        assert np.array_equal(oracle.ws_select(f, y, alpha, C, q), _lex_select(f, y, alpha, C, q)), q


def test_ws_select_first_round():
    """From a = 0 every f is -y: B is the q/2 lowest-indexed +1 samples, then the q/2
    lowest-indexed -1 samples."""
    X, y = synth.two_blobs(300, 4, seed=9)
    r = oracle.train_ws(X, y, 1.0, 0.5, 1e-3, 16, ws_trace_len=1)
    expect = np.concatenate([np.flatnonzero(y == 1)[:8], np.flatnonzero(y == -1)[:8]])
    assert np.array_equal(r.ws_trace[0], expect)


@pytest.mark.parametrize("q", [4, 16, 64, 256])
def test_ws_same_optimum(q):
    """Any working-set size reaches the optimum the pair steps reach: KKT to tol with f
    recomputed from alpha through the kernel directly, the equality constraint, the box,
    and the dual objective of the maximal-violating-pair solution."""
    wl = synth.workload(0)
    X, y, _, _ = synth.generate(0)
    ref = oracle.train(X, y, wl.C, wl.gamma, wl.tol)
    r = oracle.train_ws(X, y, wl.C, wl.gamma, wl.tol, q, want_f=True)
    assert r.status == 0 and r.rounds >= 1
    assert abs(float(r.alpha @ y)) <= 1e-10 * wl.C * X.shape[0]
    assert r.alpha.min() >= 0.0 and r.alpha.max() <= wl.C
    f = oracle.f_from_alpha(X, y, r.alpha, wl.gamma)
    np.testing.assert_allclose(r.f, f, atol=1e-9)
    up = ((y > 0) & (r.alpha < wl.C)) | ((y < 0) & (r.alpha > 0))
    low = ((y > 0) & (r.alpha > 0)) | ((y < 0) & (r.alpha < wl.C))
    assert f[low].max() - f[up].min() <= wl.tol + 1e-9
    assert abs(r.dual_obj - ref.dual_obj) <= 1e-6 * abs(ref.dual_obj)


@pytest.mark.parametrize("seed", range(20))
def test_ws_bruteforce_qp(seed):
    n = 3 + seed % 8  # 3..10
    X, y, gamma, C = _tiny_problem(seed + 500, n)
    K = rbf(X, X, gamma)
    Q = (y[:, None] * y[None, :]) * K
    a_star, _, _, _ = bf.solve(Q, y, C)
    r = oracle.train_ws(X, y, C, gamma, 1e-11, 4)
    assert r.status == 0
    np.testing.assert_allclose(r.alpha, a_star, atol=1e-6)
    assert abs(r.dual_obj - dual_W(K, y, a_star)) <= 1e-9 * max(1.0, abs(r.dual_obj))


def test_ws_invariants_between_rounds():
    """Cut after any number of steps (mid-round included): the round's change is applied
    in full, so alpha stays feasible and f equals its definition."""
    X, y = synth.two_blobs(200, 5, seed=4)
    C, gamma = 1.0, 0.3
    for t in (1, 5, 17, 40, 90):
        r = oracle.train_ws(X, y, C, gamma, 1e-3, 16, max_iter=t, want_f=True)
        assert r.iterations <= t
        assert abs(float(r.alpha @ y)) <= 1e-12 * 200
        assert r.alpha.min() >= 0.0 and r.alpha.max() <= C
        np.testing.assert_allclose(r.f, oracle.f_from_alpha(X, y, r.alpha, gamma), atol=1e-10)
