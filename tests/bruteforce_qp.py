"""Exact solution of the SVM dual QP for tiny n by active-set enumeration.

An independent pin for the oracle: it does not iterate, it enumerates every
assignment of each multiplier to {at 0, at C, free} (3^n of them), solves the
KKT equality system on the free set, and accepts the assignment whose solution is
feasible and whose bound multipliers carry the right signs.  For a positive
definite Q (RBF Gram of distinct points) the optimum is unique.

Dual (the training QP of the paper, Section III.A/III.B, in its standard form):
    min 1/2 a^T Q a - 1^T a   s.t.  y^T a = 0,  0 <= a <= C,   Q_ij = y_i y_j K_ij
KKT with multiplier nu of the equality: g = Q a - 1 + nu y,
    g_i >= 0 where a_i = 0,  g_i <= 0 where a_i = C,  g_i = 0 where 0 < a_i < C.
The bias of d(x) = sum a_i y_i K(x_i, x) - b is b = -nu.
"""
from __future__ import annotations

import itertools

import numpy as np


def solve(Q: np.ndarray, y: np.ndarray, C: float, feas_tol=1e-10, kkt_tol=1e-9):
    """Return (alpha, b, n_accepted, has_free) of the exact optimum.

    Without a free multiplier b is only fixed to an interval; the midpoint of
    that interval is returned and ``has_free`` is False."""
    n = Q.shape[0]
    y = y.astype(np.float64)
    best = None
    accepted = 0
    for states in itertools.product((0, 1, 2), repeat=n):
        st = np.array(states)
        F = np.flatnonzero(st == 2)
        U = np.flatnonzero(st == 1)
        alpha = np.zeros(n)
        alpha[U] = C
        if F.size:
            k = F.size
            A = np.zeros((k + 1, k + 1))
            A[:k, :k] = Q[np.ix_(F, F)]
            A[:k, k] = y[F]
            A[k, :k] = y[F]
            rhs = np.empty(k + 1)
            rhs[:k] = 1.0 - C * Q[np.ix_(F, U)].sum(axis=1)
            rhs[k] = -C * y[U].sum()
            try:
                sol = np.linalg.solve(A, rhs)
            except np.linalg.LinAlgError:
                continue
            if not np.all(np.isfinite(sol)):
                continue
            aF, nu = sol[:k], sol[k]
            if np.any(aF < -feas_tol) or np.any(aF > C + feas_tol):
                continue
            alpha[F] = np.clip(aF, 0.0, C)
            g = Q @ alpha - 1.0 + nu * y
            Z = np.flatnonzero(st == 0)
            if np.any(g[Z] < -kkt_tol) or np.any(g[U] > kkt_tol):
                continue
        else:
            if abs(y[U].sum()) > 0.5:  # y^T a = C * sum_U y must vanish
                continue
            h = Q @ alpha - 1.0  # g = h + nu y
            lo, hi = -np.inf, np.inf
            for i in range(n):
                # at 0: h_i + nu y_i >= 0 ; at C: h_i + nu y_i <= 0
                sgn = 1.0 if st[i] == 0 else -1.0
                # sgn * (h_i + nu y_i) >= 0  ->  sgn*y_i*nu >= -sgn*h_i
                c = sgn * y[i]
                r = -sgn * h[i]
                if c > 0:
                    lo = max(lo, r / c)
                else:
                    hi = min(hi, r / c)
            if lo > hi + kkt_tol:
                continue
            nu = 0.5 * (lo + hi) if np.isfinite(lo) and np.isfinite(hi) else (lo if np.isfinite(lo) else hi)
        accepted += 1
        if best is None:
            best = (alpha.copy(), -nu, bool(F.size))
    if best is None:
        raise RuntimeError("no KKT point found")
    return best[0], best[1], accepted, best[2]


def rbf_gram(X: np.ndarray, gamma: float) -> np.ndarray:
    X = X.astype(np.float64)
    d2 = ((X[:, None, :] - X[None, :, :]) ** 2).sum(-1)
    return np.exp(-gamma * d2)


def dual_objective(K: np.ndarray, y: np.ndarray, alpha: np.ndarray) -> float:
    v = alpha * y
    return float(alpha.sum() - 0.5 * v @ K @ v)
