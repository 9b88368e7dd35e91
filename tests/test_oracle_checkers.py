"""Pins of the oracle functions the GPU gates are judged by (no GPU).

The GPU parity tests compare the HIP library against four oracle routines besides the
solvers: the kernel rows (the 1e-5 row and Gram gates), the decision values (the 1e-3
decision gate), f recomputed from alpha for a list of rows (every full-size KKT check)
and the per-round margin of the working-set oracle (the comparison window of every
working-set trace), plus the one-vs-one vote.  Each is checked here against an
independent route: SciPy distances with NumPy fp64 sums, a plain NumPy re-derivation of
the working-set rounds, and hand-built vote tables.  A planted mistake (a row offset, a
missing bias, rows[q] read as q, a dropped margin term) fails at least one test.
"""
import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
from paper_2311_14908_amd import synth


def rbf(X, Z, gamma):
    return np.exp(-gamma * cdist(X.astype(np.float64), Z.astype(np.float64), "sqeuclidean"))


def _data(seed, n, d):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, d)).astype(np.float32)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int32)
    y[0], y[1] = 1, -1
    return X, y


# --- kernel rows (Section III.A; RBF of Section III.C) ---------------------------------

@pytest.mark.parametrize("n,d,gamma", [(37, 3, 0.7), (513, 16, 1 / 16), (300, 784, 0.02)])
def test_kernel_rows_against_scipy(n, d, gamma):
    X, _ = _data(n + d, n, d)
    rng = np.random.default_rng(1)
    # first, last, duplicates and a random spread
    rows = np.concatenate([[0, n - 1, n - 1, 0], rng.integers(0, n, 12)]).astype(np.int64)
    got = oracle.kernel_rows(X, rows, gamma)
    ref = rbf(X[rows], X, gamma)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=0)
    # K(x, x) = 1 exactly on the diagonal positions
    assert np.all(got[np.arange(rows.size), rows] == 1.0)
    # a row offset by one (a plausible indexing mistake) is far outside the tolerance
    off = rbf(X[np.minimum(rows + 1, n - 1)], X, gamma)
    assert np.max(np.abs(off - got) / ref) > 1e-3


def test_kernel_rows_linear_kind():
    X, _ = _data(5, 50, 7)
    rows = np.array([3, 49, 0, 3], dtype=np.int64)
    got = oracle.kernel_rows(X, rows, 0.0, kind=oracle.LINEAR)
    np.testing.assert_allclose(got, X[rows].astype(np.float64) @ X.astype(np.float64).T, rtol=1e-12, atol=1e-12)


def test_kernel_rows_thread_count_invariant():
    X, _ = _data(9, 400, 32)
    rows = np.arange(0, 400, 37, dtype=np.int64)
    a = oracle.kernel_rows(X, rows, 0.1, threads=1)
    b = oracle.kernel_rows(X, rows, 0.1, threads=8)
    assert np.array_equal(a, b)


# --- decision values d(x) = sum_{a_i>0} a_i y_i K(x_i, x) - b ----------------------------

@pytest.mark.parametrize("n,d,m", [(60, 4, 25), (700, 32, 130)])
def test_decision_against_numpy(n, d, m):
    X, y = _data(n, n, d)
    rng = np.random.default_rng(n + 1)
    T = rng.standard_normal((m, d)).astype(np.float32)
    alpha = rng.uniform(0.0, 2.0, n)
    alpha[rng.random(n) < 0.4] = 0.0  # non-support vectors contribute nothing
    b = 0.318
    gamma = 0.4
    got = oracle.decision(X, y, alpha, b, T, gamma)
    ref = rbf(T, X, gamma) @ (alpha * y) - b
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10)
    # the bias is subtracted: leaving it out moves every value by b
    assert np.min(np.abs((ref + b) - got)) > 0.3


def test_decision_sign_convention():
    """With every multiplier zero d(x) = -b; the label is +1 iff d > 0."""
    X, y = _data(3, 20, 2)
    T = np.zeros((3, 2), np.float32)
    for b in (-0.5, 0.0, 0.5):
        d = oracle.decision(X, y, np.zeros(20), b, T, 1.0)
        assert np.all(d == -b)


# --- f recomputed from alpha for a list of rows ------------------------------------------

def test_f_from_alpha_rows_against_numpy():
    X, y = _data(17, 400, 12)
    rng = np.random.default_rng(17)
    alpha = rng.uniform(0.0, 1.0, 400)
    alpha[rng.random(400) < 0.5] = 0.0
    gamma = 0.3
    rows = rng.permutation(400)[:90].astype(np.int64)
    rows = np.concatenate([rows, rows[:5], [0, 399]]).astype(np.int64)  # duplicates, both ends
    got = oracle.f_from_alpha(X, y, alpha, gamma, rows=rows)
    K = rbf(X, X, gamma)
    ref = K[rows] @ (alpha * y) - y[rows]
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-11)
    # the listed rows are rows[q], not q: the full vector indexed by rows gives the same bits
    full = oracle.f_from_alpha(X, y, alpha, gamma)
    assert np.array_equal(got, full[rows])
    # reading row q instead of rows[q] would be caught
    wrong = K[: rows.size] @ (alpha * y) - y[: rows.size]
    assert np.max(np.abs(wrong - got)) > 1e-2


# --- working-set rounds: the per-round margin ----------------------------------------------

def _ws_reference(X, y, C, gamma, tol, q, frac, max_inner, max_iter):
    """The working-set rounds restated with NumPy (same reading as the oracle: B from the
    ranked lists, pair steps on B until max(tol, frac x gap), f updated from B's change), and
    the margin of every round: the smallest distance of one of its decisions from flipping --
    the stop test, the two lists' boundaries at q/2, every pair selection against every other
    candidate, every local stop test and every new multiplier against its box."""
    n = X.shape[0]
    # the kernel values themselves are the oracle's (pinned above against SciPy), so that the
    # rounds take the same decisions where a margin is within rounding of zero
    K = oracle.kernel_rows(X, np.arange(n), gamma)
    yf = y.astype(np.float64)
    alpha = np.zeros(n)
    f = -yf.copy()
    idx = np.arange(n)

    def sets(a):
        up = ((y > 0) & (a < C)) | ((y < 0) & (a > 0))
        low = ((y > 0) & (a > 0)) | ((y < 0) & (a < C))
        return up, low

    out = []
    t = 0
    rnd = 0
    while True:
        up, low = sets(alpha)
        if not up.any() or not low.any():
            break
        iu = idx[up][np.lexsort((idx[up], f[up]))]
        il = idx[low][np.lexsort((idx[low], -f[low]))]
        u, l = int(iu[0]), int(il[0])
        gap = f[l] - f[u]
        margins = [abs(gap - tol)]
        rec = {"u": u, "l": l, "b_up": f[u], "b_low": f[l], "t": t}
        out.append(rec)
        if gap <= tol or t >= max_iter:
            rec["margin"] = margins[0]
            break
        h = q // 2
        B = list(iu[:h])
        B += [int(v) for v in il[:h] if v not in set(B)]
        B = np.array(B, dtype=np.int64)
        if rnd > 0 and iu.size > h:
            margins.append(f[iu[h]] - f[iu[h - 1]])
        if rnd > 0 and il.size > h:
            margins.append(f[il[h - 1]] - f[il[h]])
        m = B.size
        KB = K[np.ix_(B, B)]
        fB = f[B].copy()
        aB = alpha[B].copy()
        yB = y[B]
        tol_loc = max(tol, frac * gap)
        for inner in range(max_inner):
            if t >= max_iter:
                break
            upB = ((yB > 0) & (aB < C)) | ((yB < 0) & (aB > 0))
            lowB = ((yB > 0) & (aB > 0)) | ((yB < 0) & (aB < C))
            pos = np.arange(m)
            pu = pl = -1
            if upB.any():
                cand = pos[upB]
                pu = int(cand[np.lexsort((B[cand], fB[cand]))][0])
            if lowB.any():
                cand = pos[lowB]
                pl = int(cand[np.lexsort((B[cand], -fB[cand]))][0])
            if pu >= 0 and pl >= 0:
                margins.append(abs((fB[pl] - fB[pu]) - tol_loc))
                if not (rnd == 0 and inner == 0):
                    for a in range(m):
                        if a != pu and upB[a]:
                            margins.append(abs(fB[a] - fB[pu]))
                        if a != pl and lowB[a]:
                            margins.append(abs(fB[pl] - fB[a]))
            if pu < 0 or pl < 0 or fB[pl] - fB[pu] <= tol_loc:
                break
            eta = KB[pu, pu] + KB[pl, pl] - 2.0 * KB[pu, pl]
            if eta <= 0.0:
                eta = 1e-12
            yu, yl = float(yB[pu]), float(yB[pl])
            s = yu * yl
            au, al = aB[pu], aB[pl]
            if s < 0:
                L, H = max(0.0, al - au), min(C, C + al - au)
            else:
                L, H = max(0.0, au + al - C), min(C, au + al)
            raw = al + yl * (fB[pu] - fB[pl]) / eta
            margins.append(min(abs(raw - L), abs(raw - H)) / C)
            al_new = min(max(raw, L), H)
            au_new = min(max(au + s * (al - al_new), 0.0), C)
            snap = 1e-12 * C
            al_new = 0.0 if abs(al_new) <= snap else (C if abs(al_new - C) <= snap else al_new)
            au_new = 0.0 if abs(au_new) <= snap else (C if abs(au_new - C) <= snap else au_new)
            cu, cl = (au_new - au) * yu, (al_new - al) * yl
            fB = fB + (cu * KB[pu] + cl * KB[pl])
            aB[pu], aB[pl] = au_new, al_new
            t += 1
        c = (aB - alpha[B]) * yf[B]
        s_acc = np.zeros(n)
        for a in range(m):
            if c[a] != 0.0:
                s_acc = s_acc + c[a] * K[B[a]]
        f = f + s_acc
        alpha[B] = aB
        rec["margin"] = min(margins)
        rnd += 1
    return out, alpha


@pytest.mark.parametrize("seed,q", [(0, 4), (1, 4), (2, 6), (3, 8)])
def test_ws_trace_margin_against_reference(seed, q):
    X, y = synth.two_blobs(70, 3, seed=40 + seed)
    C, gamma, tol = 1.0, 0.5, 1e-3
    ref, a_ref = _ws_reference(X, y, C, gamma, tol, q, oracle.WS_FRAC, oracle.WS_INNER_PER_Q * q, 10**7)
    r = oracle.train_ws(X, y, C, gamma, tol, q, trace_len=len(ref) + 5)
    assert r.rounds + 1 == len(ref)
    assert np.array_equal(r.trace_ul, np.array([[e["u"], e["l"]] for e in ref], dtype=np.int32))
    assert np.array_equal(r.trace_t, np.array([e["t"] for e in ref]))
    np.testing.assert_allclose(r.trace_b, np.array([[e["b_up"], e["b_low"]] for e in ref]), atol=1e-11, rtol=0)
    np.testing.assert_allclose(r.trace_margin, np.array([e["margin"] for e in ref]), atol=1e-11, rtol=0)
    np.testing.assert_allclose(r.alpha, a_ref, atol=1e-11, rtol=0)
    # the margins are sharp: dropping the box-distance term (a plausible omission) changes them
    assert np.any(r.trace_margin[:-1] < 0.05)


# --- one-vs-one vote --------------------------------------------------------------------

def _zero_models(labels, k, biases):
    """One-vs-one models whose multipliers are all zero, so that d = -b for every point."""
    out = []
    for (a, b), bias in zip(oracle.ovo_pairs(k), biases):
        idx, y = oracle.ovo_local(labels, a, b)
        r = oracle.TrainResult(alpha=np.zeros(idx.size), b=bias, b_up=bias, b_low=bias, dual_obj=0.0,
                               iterations=0, n_sv=0, n_bound=0, status=0)
        out.append((idx, y, r))
    return out


def test_ovo_vote_three_way_tie_goes_to_smallest_class():
    X, lab = synth.multiclass_blobs(30, 2, 3, seed=1)
    T = np.zeros((4, 2), np.float32)
    # pairs (0,1), (0,2), (1,2): 0 beats 1, 2 beats 0, 1 beats 2 -> one vote each
    models = _zero_models(lab, 3, [-1.0, 1.0, -1.0])
    dec, pred = oracle.predict_ovo(X, lab, 3, models, T, 1.0)
    np.testing.assert_array_equal(dec, np.tile([1.0, -1.0, 1.0], (4, 1)))
    np.testing.assert_array_equal(pred, [0, 0, 0, 0])


def test_ovo_vote_tie_between_later_classes():
    X, lab = synth.multiclass_blobs(40, 2, 4, seed=2)
    T = np.zeros((2, 2), np.float32)
    # pairs (0,1) (0,2) (0,3) (1,2) (1,3) (2,3): 1 beats 0, 2 beats 0, 0 beats 3, 2 beats 1,
    # 1 beats 3, 3 beats 2 -> votes 0:1, 1:2, 2:2, 3:1 -> class 1 (the smaller of the tie)
    models = _zero_models(lab, 4, [1.0, 1.0, -1.0, 1.0, -1.0, 1.0])
    _, pred = oracle.predict_ovo(X, lab, 4, models, T, 1.0)
    np.testing.assert_array_equal(pred, [1, 1])


def test_ovo_vote_zero_decision_votes_for_b():
    """d = 0 is not > 0, so pair (a, b) votes b."""
    X, lab = synth.multiclass_blobs(20, 2, 2, seed=3)
    T = np.zeros((3, 2), np.float32)
    _, pred = oracle.predict_ovo(X, lab, 2, _zero_models(lab, 2, [0.0]), T, 1.0)
    np.testing.assert_array_equal(pred, [1, 1, 1])
    _, pred = oracle.predict_ovo(X, lab, 2, _zero_models(lab, 2, [-1e-300]), T, 1.0)
    np.testing.assert_array_equal(pred, [0, 0, 0])
