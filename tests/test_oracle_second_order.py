"""Pins of the oracle's second-order selection (oracle.train(..., selection=SECOND_ORDER), no GPU).

The paper cites two working-pair rules for SMO (Section III.B); besides the maximal violating
pair the oracle implements the second-order rule for the second index: u = argmin_{I_up} f,
l = argmax over t in I_low with f_t > f_u of (f_t - f_u)^2 / a_ut, a_ut = K_uu + K_tt - 2 K_ut.
Pinned against: the rule re-evaluated by brute force with SciPy kernel values at sampled steps,
the first step in closed form, invariants after every step, the exact optimum of enumerated
problems, the KKT / duality-gap certificate, and LIBSVM (which uses a rule of this kind) as a
loose external count.
"""
import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
from paper_2311_14908_amd import synth
from tests import bruteforce_qp as bf

SO = oracle.SECOND_ORDER


def rbf(X, Z, gamma):
    return np.exp(-gamma * cdist(X.astype(np.float64), Z.astype(np.float64), "sqeuclidean"))


def dual_W(K, y, a):
    v = a * y
    return float(a.sum() - 0.5 * v @ K @ v)


def sets(y, a, C):
    up = ((y > 0) & (a < C)) | ((y < 0) & (a > 0))
    low = ((y > 0) & (a > 0)) | ((y < 0) & (a < C))
    return up, low


def test_selection_is_the_second_order_rule():
    """At sampled steps the pair is (argmin_{I_up} f, argmax of the gain over I_low above f_u),
    both re-evaluated from alpha with SciPy kernel values; the stop values are the first-order
    extremes."""
    X, y = synth.two_blobs(150, 4, seed=12)
    C, gamma = 0.8, 0.3
    K = rbf(X, X, gamma)
    full = oracle.train(X, y, C, gamma, 1e-3, trace_len=10_000, selection=SO)
    checked = 0
    for t in [0, 1, 2, 3, 7, 19, full.iterations // 3, full.iterations // 2, full.iterations - 1]:
        r = oracle.train(X, y, C, gamma, 1e-3, max_iter=t, selection=SO)
        a = r.alpha
        f = K @ (a * y) - y
        up, low = sets(y, a, C)
        iu = np.flatnonzero(up)[np.argmin(f[up])]
        cand = np.flatnonzero(low & (f > f[iu]))
        at = K[iu, iu] + np.diag(K)[cand] - 2.0 * K[iu, cand]
        at = np.where(at <= 0, 1e-12, at)
        g = (f[cand] - f[iu]) ** 2 / at
        best = cand[np.argmax(g)]
        # skip steps whose best two gains are within rounding of each other
        gs = np.sort(g)[::-1]
        if gs.size > 1 and (gs[0] - gs[1]) < 1e-9 * gs[0]:
            continue
        assert tuple(full.trace_ul[t]) == (iu, best), t
        np.testing.assert_allclose(full.trace_b[t], [f[iu], f[low].max()], atol=1e-10)
        checked += 1
    assert checked >= 7


def test_first_step_closed_form():
    """From a = 0 (f = -y): u is the first +1 sample; every -1 sample has f_t - f_u = 2, so l is
    the -1 sample nearest to x_u (largest K_ut); both multipliers move to min(C, 2/eta)."""
    for cid in (0, 2, 3):
        wl = synth.workload(cid)
        X, y, _, _ = synth.generate(cid, n=300, m=1)
        r = oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=1, trace_len=2, selection=SO)
        u = int(np.flatnonzero(y == 1)[0])
        neg = np.flatnonzero(y == -1)
        k = rbf(X[u:u + 1], X[neg], wl.gamma)[0]
        l = int(neg[np.argmax(k)])
        assert tuple(r.trace_ul[0]) == (u, l)
        eta = 2.0 - 2.0 * k.max()
        a1 = min(wl.C, 2.0 / eta)
        np.testing.assert_allclose([r.alpha[u], r.alpha[l]], [a1, a1], rtol=1e-12)
        assert np.count_nonzero(r.alpha) == 2


def test_invariants_every_step():
    X, y = synth.two_blobs(120, 5, seed=3)
    C, gamma = 1.0, 0.2
    K = rbf(X, X, gamma)
    full = oracle.train(X, y, C, gamma, 1e-3, selection=SO)
    prev = -np.inf
    for t in range(1, full.iterations + 1):
        r = oracle.train(X, y, C, gamma, 1e-3, max_iter=t, want_f=True, selection=SO)
        a = r.alpha
        assert abs(float(a @ y)) <= 1e-10 * C * len(y)
        assert np.all(a >= 0.0) and np.all(a <= C)
        np.testing.assert_allclose(r.f, K @ (a * y) - y, atol=1e-9)
        W = dual_W(K, y, a)
        assert W > prev
        prev = W


def _tiny_problem(seed, n):
    rng = np.random.default_rng(seed)
    d = int(rng.integers(2, 6))
    X = rng.standard_normal((n, d)).astype(np.float32)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int32)
    y[0], y[1] = 1, -1
    return X, y, float(rng.uniform(0.1, 1.5)), float(rng.choice([0.3, 1.0, 5.0, 100.0]))


@pytest.mark.parametrize("seed", range(24))
def test_bruteforce_qp(seed):
    n = 3 + seed % 8
    X, y, gamma, C = _tiny_problem(seed + 900, n)
    K = rbf(X, X, gamma)
    Q = (y[:, None] * y[None, :]) * K
    a_star, _, _, _ = bf.solve(Q, y, C)
    r = oracle.train(X, y, C, gamma, 1e-11, selection=SO)
    assert r.status == 0
    np.testing.assert_allclose(r.alpha, a_star, atol=1e-6)
    assert abs(r.dual_obj - dual_W(K, y, a_star)) <= 1e-9 * max(1.0, abs(r.dual_obj))


@pytest.mark.parametrize("cid", [0, 2, 3])
def test_kkt_duality_gap_and_same_optimum(cid):
    wl = synth.workload(cid)
    X, y, _, _ = synth.generate(cid, n=600, m=1)
    r = oracle.train(X, y, wl.C, wl.gamma, wl.tol, selection=SO)
    mvp = oracle.train(X, y, wl.C, wl.gamma, wl.tol)
    assert r.status == 0
    K = rbf(X, X, wl.gamma)
    a = r.alpha
    f = K @ (a * y) - y
    up, low = sets(y, a, wl.C)
    assert np.all(f[up] >= r.b - wl.tol / 2 - 1e-9)
    assert np.all(f[low] <= r.b + wl.tol / 2 + 1e-9)
    W = dual_W(K, y, a)
    v = a * y
    P = 0.5 * v @ K @ v + wl.C * np.maximum(0.0, 1.0 - y * (K @ v - r.b)).sum()
    assert -1e-9 <= P - W <= len(y) * wl.C * wl.tol
    assert abs(W - mvp.dual_obj) <= 1e-4 * abs(mvp.dual_obj)


def test_fewer_steps_than_the_maximal_violating_pair_and_close_to_libsvm():
    """LIBSVM (through scikit-learn, shrinking off) selects with second-order information too;
    its trajectory differs in tie-breaks and rounding, so only the step counts are compared:
    within 15% of each other, and both below the maximal violating pair's."""
    from sklearn.svm import SVC
    for seed in range(4):
        X, y = synth.two_blobs(300 + 50 * seed, 5, seed=seed)
        C, g, tol = [0.5, 1.0, 10.0, 1.0][seed], 0.3, 1e-3
        so = oracle.train(X, y, C, g, tol, selection=SO)
        mvp = oracle.train(X, y, C, g, tol)
        sk = SVC(kernel="rbf", C=C, gamma=g, tol=tol, shrinking=False).fit(X.astype(np.float64), y)
        n_sk = int(np.atleast_1d(sk.n_iter_)[0])
        assert abs(so.iterations - n_sk) <= 0.15 * n_sk, (seed, so.iterations, n_sk)
        assert so.iterations < mvp.iterations and n_sk < mvp.iterations


def test_rejects_unknown_selection():
    X, y = synth.two_blobs(20, 2, seed=1)
    with pytest.raises(ValueError):
        oracle.train(X, y, 1.0, 0.5, 1e-3, selection=2)
