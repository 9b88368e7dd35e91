"""Label and validity checks shared by the GPU tests (plain NumPy on the oracle's values).

Labels are compared on every test point.  A binary label may differ from the oracle's only
where the oracle's decision value lies within the measured decision error of zero (there the
fp32 kernel values can move it across), and every such point is reported.  For one-vs-one the
predicted class must be one the votes allow: the pair decisions within the error of zero may
fall either way, every combination is enumerated, and a point whose decisions are all clear of
zero must get exactly the oracle's class.
"""
import itertools

import numpy as np


def check_binary_labels(d_gpu, d_ref, err):
    """Every point: identical labels, except where |d_ref| <= err (reported).  Returns the
    number of points that differ."""
    d_gpu, d_ref = np.asarray(d_gpu), np.asarray(d_ref)
    differ = (d_gpu > 0) != (d_ref > 0)
    near = np.abs(d_ref) <= err
    if differ.any():
        print(f"labels differ at {int(differ.sum())} of {d_ref.size} points, |d_oracle| = "
              f"{np.abs(d_ref[differ]).tolist()} (decision error {err:.2e})")
    assert not np.any(differ & ~near), "a label differs where the oracle's decision is clear of zero"
    assert int(differ.sum()) <= int(near.sum())
    return int(differ.sum())


_PAIRS = {}


def _pairs(k):
    if k not in _PAIRS:
        ab = np.array([(a, b) for a in range(k) for b in range(a + 1, k)], np.int64)
        _PAIRS[k] = (ab[:, 0], ab[:, 1])
    return _PAIRS[k]


def ovo_vote(signs, k):
    """Class voted by one test point: pair (a<b) in lexicographic order votes a iff its decision is
    positive, else b; most votes wins, ties to the smaller class."""
    a, b = _pairs(k)
    votes = np.bincount(np.where(np.asarray(signs, bool), a, b), minlength=k)
    return int(np.argmax(votes))  # the first (smallest) class on ties


def ovo_allowed_classes(dec_row, k, err, max_free=12):
    """The classes the votes can give when the pair decisions within err of zero fall either way
    (all of them enumerated; None if more than max_free are that close)."""
    dec_row = np.asarray(dec_row)
    free = np.flatnonzero(np.abs(dec_row) <= err)
    if free.size > max_free:
        return None
    base = dec_row > 0
    out = set()
    for flips in itertools.product([False, True], repeat=free.size):
        s = base.copy()
        s[free] = np.array(flips, bool) if free.size else s[free]
        out.add(ovo_vote(s, k))
    return out


def check_ovo_predictions(pred_gpu, dec_ref, k, err):
    """Every point: the GPU's class must be one the oracle's decisions allow (exactly the
    oracle's where no pair decision is within err of zero).  Returns the number of points whose
    class was not determined."""
    pred_gpu = np.asarray(pred_gpu)
    ambiguous = 0
    for i in range(dec_ref.shape[0]):
        allowed = ovo_allowed_classes(dec_ref[i], k, err)
        assert allowed is not None, f"point {i}: too many pair decisions near zero to enumerate"
        if len(allowed) > 1:
            ambiguous += 1
        assert int(pred_gpu[i]) in allowed, (i, int(pred_gpu[i]), sorted(allowed))
    if ambiguous:
        print(f"{ambiguous} of {dec_ref.shape[0]} points have a class the near-zero pair decisions leave open")
    return ambiguous


def kkt_and_gap(f, y, a, b, C, tol, slack):
    """tol-KKT on every row with f recomputed from alpha, and the duality-gap certificate
    0 <= P - W <= n C tol, P = 1/2 a'Qa + C sum max(0, 1 - y_i d_i), d_i = f_i + y_i - b."""
    f, y, a = np.asarray(f, np.float64), np.asarray(y, np.float64), np.asarray(a, np.float64)
    up = ((y > 0) & (a < C)) | ((y < 0) & (a > 0))
    low = ((y > 0) & (a > 0)) | ((y < 0) & (a < C))
    assert np.all(f[up] >= b - tol / 2 - slack), float(np.min(f[up] - b))
    assert np.all(f[low] <= b + tol / 2 + slack), float(np.max(f[low] - b))
    aQa = float(np.sum(a * y * (f + y)))
    W = float(a.sum()) - 0.5 * aQa
    P = 0.5 * aQa + C * float(np.sum(np.maximum(0.0, 1.0 - y * (f + y - b))))
    gap = P - W
    assert -1e-9 * abs(W) <= gap <= len(y) * C * tol, (gap, W)
    return gap, W
