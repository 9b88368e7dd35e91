"""Seeded synthetic workloads for the binary and one-vs-one RBF-SVM solves.

This module only draws inputs. It holds none of the SVM arithmetic (no kernel,
no dual, no SMO) so that the CPU oracle and the HIP path can both be fed from it
without sharing any of the method's code.

The paper measures on Pavia Centre, Iris and Breast Cancer Wisconsin
(Section IV.A, Table 1). None of them is used here; these five synthetic
workloads stand in for them at larger sample counts:

  id  shape                      recipe
  0   n=1,000    d=16   binary   two isotropic blobs, means +-0.5*1, sigma 1, balanced
  1   n=20,000   d=784  binary   U[0,1] features, 80% zeroed; label = sign of a random
                                 projection centred at its median; 5% flips
  2   n=50,000   d=128  binary   8-component mixture (4 per class), means ~ N(0,4I), sigma 1,
                                 5% flips
  3   n=100,000  d=32   binary   two overlapping blobs, means +-0.3*1, sigma 1
  4   n=60,000   d=784  10-class one-vs-one; class means ~ N(0,I); x = clip(mean + N(0,0.25 I), 0, 1)

Every generator takes ``n`` (and ``m`` test points) so that tests can draw the
same recipe at reduced size.  Arrays are C-contiguous: X float32 [n, d];
y int32 in {-1, +1} for binary workloads, labels int32 in 0..k-1 for one-vs-one.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    """Sizes and hyper-parameters of one synthetic workload."""
    cid: int
    name: str
    n: int
    d: int
    C: float
    gamma: float
    tol: float
    classes: int  # 2 for binary, k for one-vs-one
    m_test: int


WORKLOADS = (
    Workload(0, "blobs-n1000-d16", 1_000, 16, 1.0, 1.0 / 16, 1e-3, 2, 1_000),
    Workload(1, "sparse-proj-n20000-d784", 20_000, 784, 10.0, 0.02, 1e-3, 2, 10_000),
    Workload(2, "mixture8-n50000-d128", 50_000, 128, 10.0, 1.0 / 128, 1e-3, 2, 10_000),
    Workload(3, "blobs-n100000-d32", 100_000, 32, 1.0, 1.0 / 32, 1e-3, 2, 10_000),
    Workload(4, "ovo10-n60000-d784", 60_000, 784, 10.0, 0.02, 1e-3, 10, 10_000),
)


def workload(cid: int) -> Workload:
    return WORKLOADS[cid]


def _flip(rng: np.random.Generator, y: np.ndarray, frac: float) -> np.ndarray:
    """Flip the sign of exactly round(frac*n) labels chosen without replacement."""
    y = y.copy()
    k = int(round(frac * y.shape[0]))
    if k:
        idx = rng.choice(y.shape[0], size=k, replace=False)
        y[idx] = -y[idx]
    return y


def _balanced_signs(rng: np.random.Generator, n: int) -> np.ndarray:
    y = np.where(np.arange(n) < (n + 1) // 2, 1, -1).astype(np.int32)
    return y[rng.permutation(n)]


def _blobs(rng, n, d, shift, balanced):
    y = _balanced_signs(rng, n) if balanced else np.where(rng.random(n) < 0.5, 1, -1).astype(np.int32)
    X = rng.standard_normal((n, d)) + shift * y[:, None].astype(np.float64)
    return X.astype(np.float32), y


def _gen0(seed, n, m, d):
    rng = np.random.default_rng(seed)
    Xtr, ytr = _blobs(rng, n, d, 0.5, True)
    rt = np.random.default_rng(1000 + seed)
    Xte, yte = _blobs(rt, m, d, 0.5, True)
    return Xtr, ytr, Xte, yte


def _gen1(seed, n, m, d):
    rng = np.random.default_rng(seed)
    w = rng.standard_normal(d)

    def draw(r, k):
        X = r.random((k, d))
        X[r.random((k, d)) < 0.8] = 0.0
        return X.astype(np.float32)

    Xtr = draw(rng, n)
    ptr = Xtr.astype(np.float64) @ w
    thr = float(np.median(ptr))
    ytr = np.where(ptr - thr >= 0.0, 1, -1).astype(np.int32)
    ytr = _flip(rng, ytr, 0.05)
    rt = np.random.default_rng(1000 + seed)
    Xte = draw(rt, m)
    yte = np.where(Xte.astype(np.float64) @ w - thr >= 0.0, 1, -1).astype(np.int32)
    yte = _flip(rt, yte, 0.05)
    return Xtr, ytr, Xte, yte


def _gen2(seed, n, m, d):
    rng = np.random.default_rng(seed)
    mu = 2.0 * rng.standard_normal((8, d))
    comp_sign = np.array([1, 1, 1, 1, -1, -1, -1, -1], dtype=np.int32)

    def draw(r, k):
        comp = np.arange(k) % 8  # equal weight
        comp = comp[r.permutation(k)]
        X = mu[comp] + r.standard_normal((k, d))
        return X.astype(np.float32), comp_sign[comp].copy()

    Xtr, ytr = draw(rng, n)
    ytr = _flip(rng, ytr, 0.05)
    rt = np.random.default_rng(1000 + seed)
    Xte, yte = draw(rt, m)
    yte = _flip(rt, yte, 0.05)
    return Xtr, ytr, Xte, yte


def _gen3(seed, n, m, d):
    rng = np.random.default_rng(seed)
    Xtr, ytr = _blobs(rng, n, d, 0.3, False)
    rt = np.random.default_rng(1000 + seed)
    Xte, yte = _blobs(rt, m, d, 0.3, False)
    return Xtr, ytr, Xte, yte


def _gen4(seed, n, m, d, k=10):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((k, d))

    def draw(r, cnt):
        lab = np.arange(cnt) % k  # equal class sizes
        lab = lab[r.permutation(cnt)].astype(np.int32)
        X = np.clip(mu[lab] + 0.5 * r.standard_normal((cnt, d)), 0.0, 1.0)
        return X.astype(np.float32), lab

    Xtr, ltr = draw(rng, n)
    rt = np.random.default_rng(1000 + seed)
    Xte, lte = draw(rt, m)
    return Xtr, ltr, Xte, lte


_GENS = (_gen0, _gen1, _gen2, _gen3, _gen4)


def generate(cid: int, n: int | None = None, m: int | None = None, d: int | None = None,
             seed: int | None = None, classes: int | None = None):
    """Draw workload ``cid`` (optionally resized).

    Returns ``(X, y, X_test, y_test)``.  ``seed`` defaults to the workload id;
    the test split uses seed ``1000 + seed``.
    """
    wl = WORKLOADS[cid]
    n = wl.n if n is None else int(n)
    m = wl.m_test if m is None else int(m)
    d = wl.d if d is None else int(d)
    seed = cid if seed is None else int(seed)
    if cid == 4:
        k = wl.classes if classes is None else int(classes)
        out = _gen4(seed, n, m, d, k)
    else:
        out = _GENS[cid](seed, n, m, d)
    return tuple(np.ascontiguousarray(a) for a in out)


def two_blobs(n: int, d: int, seed: int, shift: float = 0.5):
    """Small balanced two-blob problem (recipe of workload 0) at any size."""
    rng = np.random.default_rng(seed)
    X, y = _blobs(rng, n, d, shift, True)
    return np.ascontiguousarray(X), np.ascontiguousarray(y)


def multiclass_blobs(n: int, d: int, k: int, seed: int):
    """Small k-class problem (recipe of workload 4) at any size."""
    Xtr, ltr, _, _ = _gen4(seed, n, 1, d, k)
    return Xtr, ltr


# Paper-shaped context runs: the paper's binary and nine-class timings (Tables 3 and 4) use a
# 102-band hyperspectral scene with 200-800 training samples per class.  This recipe only
# matches that shape (d = 102, `per_class` samples of each of `classes` classes); the scene
# itself is not used.  Class mean spectra ~ 0.5 + 0.2 N(0, I); samples = mean + 0.1 N(0, I),
# clipped to [0, 1].  C = 10, gamma = 0.5, tol = 1e-3 (the paper states none of them).
PAPER_SHAPE = dict(d=102, C=10.0, gamma=0.5, tol=1e-3)


def paper_shaped(per_class: int, classes: int, seed: int = 0):
    """Returns (X float32 [classes*per_class, 102], labels int32 in 0..classes-1), shuffled."""
    d = PAPER_SHAPE["d"]
    rng = np.random.default_rng(seed)
    mu = 0.5 + 0.2 * rng.standard_normal((classes, d))
    n = classes * per_class
    lab = (np.arange(n) % classes)[rng.permutation(n)].astype(np.int32)
    X = np.clip(mu[lab] + 0.1 * rng.standard_normal((n, d)), 0.0, 1.0).astype(np.float32)
    return np.ascontiguousarray(X), np.ascontiguousarray(lab)


def sparse_projection_on_device(n: int, d: int, seed: int = 1):
    """Workload 1's recipe drawn on the current GPU with torch's seeded generator, for sizes at
    which drawing on the host is slow (300,000 x 784: about a minute with NumPy): entries U[0,1]
    zeroed with probability 0.8, label = sign of a random Gaussian projection about its median
    (0 counts as +1), 5% of the labels flipped.  Same distribution as ``generate(1, n=n, d=d)``,
    other values.  Returns device tensors (X float32 [n, d], y int32 [n])."""
    import torch

    g = torch.Generator(device="cuda").manual_seed(seed)
    X = torch.rand(n, d, generator=g, device="cuda")
    X.masked_fill_(torch.rand(n, d, generator=g, device="cuda") < 0.8, 0.0)
    proj = X.double() @ torch.randn(d, generator=g, device="cuda", dtype=torch.float64)
    y = torch.where(proj >= proj.median(), 1, -1).to(torch.int32)
    flip = torch.randperm(n, generator=g, device="cuda")[:round(0.05 * n)]
    y[flip] = -y[flip]
    return X, y
