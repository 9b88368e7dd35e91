"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on identical seeded inputs.

Gates (fp64 oracle vs fp32-kernel GPU path):
  kernel rows     relative error <= 1e-5 where K >= 1e-30
  f               max |f_gpu - f_oracle| <= 1e-4 after 1, 10, 100 and 1000 steps
  working set     identical (u, l) for every step of the workload-0 solve (first 1000)
  dual objective  relative error <= 1e-4
  decisions       max abs error <= 1e-3; labels compared on every point (a label may differ only
                  where the oracle's decision lies within the measured error of zero; one-vs-one:
                  the voted class must be one the oracle's decisions allow)
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2311_14908_amd import svmx, synth
from tests.label_checks import check_binary_labels, check_ovo_predictions, ovo_vote

pytestmark = pytest.mark.gpu

ROW_RTOL = 1e-5
F_ATOL = 1e-4
W_RTOL = 1e-4
DEC_ATOL = 1e-3
PRED_ATOL = 2e-4  # decisions from the same alpha, b: fp32 kernel values against the fp64 oracle


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    svmx.load()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def row_rel_err(got, ref):
    got = np.asarray(got, np.float64)
    mask = ref >= 1e-30
    return float(np.max(np.abs(got[mask] - ref[mask]) / ref[mask])) if mask.any() else 0.0


def check_decisions(d_gpu, d_ref, gate=DEC_ATOL):
    err = float(np.max(np.abs(d_gpu - d_ref)))
    assert err <= gate
    check_binary_labels(d_gpu, d_ref, err)


def check_ovo(dec, pred, dec_ref, k, pred_ref, gate=DEC_ATOL):
    # the vote restated in the checks gives the oracle's classes from its decisions
    assert [ovo_vote(r > 0, k) for r in dec_ref] == list(pred_ref)
    dec = np.asarray(dec)
    err = float(np.max(np.abs(dec - dec_ref)))
    assert err <= gate
    check_ovo_predictions(pred, dec_ref, k, err)


# --- kernel rows and the Gram ------------------------------------------------------------

@pytest.mark.parametrize("cid", [0, 1, 2, 3, 4])
def test_kernel_rows_full_size(cid):
    wl = synth.workload(cid)
    X, _, _, _ = synth.generate(cid, m=1)
    rng = np.random.default_rng(100 + cid)
    rows = np.concatenate([[0, X.shape[0] - 1], rng.integers(0, X.shape[0], 5)])
    got = svmx.svm_kernel_rows(dev(X), wl.gamma, rows).cpu().numpy()
    ref = oracle.kernel_rows(X, rows, wl.gamma)
    assert row_rel_err(got, ref) <= ROW_RTOL
    assert np.all(got[np.arange(len(rows)), rows] == 1.0)


@pytest.mark.parametrize("n,d,misalign", [(3000, 1500, 0), (2000, 301, 0), (2000, 784, 1)])
def test_row_path_wide_and_unaligned(n, d, misalign):
    """Rows wider than one register block of the GEMV (d = 1500: 375 float4 per row, more than
    4 x 64), scalar lanes (d = 301), and X that is not 16-byte aligned (scalar lanes at d = 784):
    kernel rows against the oracle, K = 1 between identical rows, and the working set of a short
    row-path training against the oracle's up to its first near-tie."""
    X, y = synth.two_blobs(n, d, seed=d)
    X[7] = X[3]  # a duplicate pair
    gamma = 1.0 / d
    buf = torch.empty(n * d + misalign, dtype=torch.float32, device="cuda")
    Xd = buf[misalign:].view(n, d)
    Xd.copy_(torch.from_numpy(X))
    assert (Xd.data_ptr() % 16 != 0) == bool(misalign)
    rows = np.array([0, 3, 7, n - 1, 1234 % n])
    got = svmx.svm_kernel_rows(Xd, gamma, rows).cpu().numpy()
    ref = oracle.kernel_rows(X, rows, gamma)
    assert row_rel_err(got, ref) <= ROW_RTOL
    assert np.all(got[np.arange(len(rows)), rows] == 1.0)
    assert got[1, 7] == 1.0 and got[2, 3] == 1.0
    r = oracle.train(X, y, 1.0, gamma, 1e-3, max_iter=300, trace_len=300)
    out = svmx.svm_train(Xd, dev(y), 1.0, gamma, 1e-3, gram=svmx.GRAM_OFF, max_iter=300, trace_len=300)
    tied = np.flatnonzero(np.asarray(r.trace_gap)[1:].min(axis=1) < 1e-6)
    k = min(r.iterations + 1, 300, int(tied[0]) + 1 if tied.size else 300)
    assert k >= 20
    np.testing.assert_array_equal(out.trace_ul[:k], r.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], r.trace_b[:k], atol=F_ATOL, rtol=0)


MFMAS = [svmx.MFMA_SPLIT_F16, svmx.MFMA_F32]


def test_row_path_largest_placement():
    """The largest problem the row path places: 256 workgroups of 512 threads with 8 samples a
    thread (n just below 2^20).  The first 40 steps against the oracle: selections, b_up/b_low
    and the multipliers they moved."""
    n, d = 1_048_000, 16
    X, y = synth.two_blobs(n, d, seed=5)
    steps = 40
    r = oracle.train(X, y, 1.0, 1.0 / d, 1e-3, max_iter=steps, trace_len=steps)
    out = svmx.svm_train(dev(X), dev(y), 1.0, 1.0 / d, 1e-3, gram=svmx.GRAM_OFF, max_iter=steps, trace_len=steps)
    assert out.status == svmx.SVM_NOT_CONVERGED and out.stats["iterations"] == steps
    tied = np.flatnonzero(np.asarray(r.trace_gap)[1:].min(axis=1) < 1e-6)
    k = min(steps, int(tied[0]) + 1 if tied.size else steps)
    np.testing.assert_array_equal(out.trace_ul[:k], r.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], r.trace_b[:k], atol=F_ATOL, rtol=0)
    if k == steps:
        np.testing.assert_allclose(out.alpha.cpu().numpy(), r.alpha, atol=1e-5, rtol=0)



def test_host_array_conveniences_are_the_device_calls():
    """svm_train_host and svm_predict_host only copy around svm_train and svm_predict: the same
    alpha, b and decision values, bit for bit."""
    X, y, Xt, _ = synth.generate(0)
    a_h, b_h, status, st = svmx.svm_train_host(X, y, C0.C, C0.gamma, C0.tol)
    out = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol)
    assert status == svmx.SVM_OK and st["iterations"] == out.stats["iterations"]
    np.testing.assert_array_equal(a_h, out.alpha.cpu().numpy())
    assert b_h == out.b
    d_h = svmx.svm_predict_host(X, y, a_h, b_h, C0.gamma, Xt)
    d = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, C0.gamma, dev(Xt)).cpu().numpy()
    np.testing.assert_array_equal(d_h, d)
    k = 4
    Xo, lab, Xto, _ = synth.generate(4, n=400, m=50, d=12, classes=k)
    a_o, b_o, s_o, _ = svmx.svm_train_ovo_host(Xo, lab, k, 1.0, 0.1, 1e-3)
    oo = svmx.svm_train_ovo(dev(Xo), dev(lab), k, 1.0, 0.1, 1e-3)
    assert s_o == svmx.SVM_OK
    np.testing.assert_array_equal(a_o, oo.alpha.cpu().numpy())
    np.testing.assert_array_equal(b_o, oo.b)
    dh, ph = svmx.svm_predict_ovo_host(Xo, lab, k, a_o, b_o, 0.1, Xto)
    dd, pd = svmx.svm_predict_ovo(dev(Xo), dev(lab), k, oo.alpha, oo.b, 0.1, dev(Xto))
    np.testing.assert_array_equal(dh, dd.cpu().numpy())
    np.testing.assert_array_equal(ph, pd.cpu().numpy())

def test_row_path_streamed_large_configuration():
    """The row path as the 300,000 x 784 measurement runs it: default options, so each
    workgroup keeps the first rows of its slice in LDS and the rest of X (940 MB, more than
    LDS, L2 and the Infinity Cache hold) streams from HBM at every step.  The first 20 steps
    against the oracle on the same bytes: selections, b_up/b_low and the multipliers moved."""
    wl = synth.workload(1)
    Xd, yd = synth.sparse_projection_on_device(300_000, 784, seed=1)
    steps = 20
    out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_OFF, max_iter=steps, trace_len=steps)
    assert out.status == svmx.SVM_NOT_CONVERGED and out.stats["iterations"] == steps
    assert out.stats["gram_used"] == 0 and out.stats["resident_rows"] > 0
    X, y = Xd.cpu().numpy(), yd.cpu().numpy()
    del Xd, yd
    r = oracle.train(X, y, wl.C, wl.gamma, wl.tol, max_iter=steps, trace_len=steps)
    tied = np.flatnonzero(np.asarray(r.trace_gap)[1:].min(axis=1) < 1e-6)
    k = min(steps, int(tied[0]) + 1 if tied.size else steps)
    assert k >= 5
    np.testing.assert_array_equal(out.trace_ul[:k], r.trace_ul[:k])
    np.testing.assert_allclose(out.trace_b[:k], r.trace_b[:k], atol=F_ATOL, rtol=0)
    if k == steps:
        np.testing.assert_allclose(out.alpha.cpu().numpy(), r.alpha, atol=1e-5, rtol=0)


@pytest.mark.parametrize("mfma", MFMAS)
@pytest.mark.parametrize("aligned", [False, True])
@pytest.mark.parametrize("cid,n,d", [(0, 1000, 16), (2, 1300, 128), (1, 700, 784), (3, 3001, 32), (0, 333, 13),
                                     (0, 129, 5)])
def test_gram_small(cid, n, d, mfma, aligned):
    """Every entry of the Gram against the oracle.  With a row pitch that is a multiple of 64 the
    kernels store the mirrored tiles as float4s (and rows of up to 128 features take the
    one-stage kernel); with n + 3 every mirrored entry is stored on its own."""
    wl = synth.workload(cid)
    X, _, _, _ = synth.generate(cid, n=n, m=1, d=d)
    ld = (n + 63) // 64 * 64 if aligned else n + 3
    G = svmx.svm_gram(dev(X), wl.gamma, ld=ld, gram_mfma=mfma).cpu().numpy()[:, :n]
    ref = oracle.kernel_rows(X, np.arange(n), wl.gamma)
    assert row_rel_err(G, ref) <= ROW_RTOL
    assert np.all(np.diag(G) == 1.0)


@pytest.mark.parametrize("mfma", MFMAS)
@pytest.mark.parametrize("cid", [1, 2, 4])
def test_gram_sampled_full_size(cid, mfma):
    wl = synth.workload(cid)
    X, _, _, _ = synth.generate(cid, m=1)
    Gd = svmx.svm_gram(dev(X), wl.gamma, gram_mfma=mfma)
    rows = np.random.default_rng(7).integers(0, X.shape[0], 6)
    got = Gd[torch.from_numpy(rows).cuda()].cpu().numpy()
    del Gd
    torch.cuda.empty_cache()
    ref = oracle.kernel_rows(X, rows, wl.gamma)
    assert row_rel_err(got, ref) <= ROW_RTOL


# --- binary training on workload 0 -------------------------------------------------------

C0 = synth.workload(0)


@pytest.fixture(scope="module")
def c0():
    X, y, Xt, yt = synth.generate(0)
    ref = oracle.train(X, y, C0.C, C0.gamma, C0.tol, trace_len=5000, want_f=True)
    return X, y, Xt, ref


@pytest.mark.parametrize("gram,wgs,mfma", [(svmx.GRAM_ON, 0, 0), (svmx.GRAM_ON, 3, 0), (svmx.GRAM_ON, 8, 0),
                                           (svmx.GRAM_ON, 0, svmx.MFMA_F32), (svmx.GRAM_ON, 8, svmx.MFMA_F32),
                                           (svmx.GRAM_OFF, 0, 0), (svmx.GRAM_OFF, 1, 0)])
def test_train_c0_trace_and_result(c0, gram, wgs, mfma):
    X, y, Xt, ref = c0
    out = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, gram=gram, workgroups=wgs, trace_len=1001,
                         gram_mfma=mfma)
    assert out.status == svmx.SVM_OK
    st = out.stats
    assert st["iterations"] == ref.iterations
    steps = min(1000, ref.iterations + 1)
    np.testing.assert_array_equal(out.trace_ul[:steps], ref.trace_ul[:steps])
    np.testing.assert_allclose(out.trace_b[:steps], ref.trace_b[:steps], atol=F_ATOL, rtol=0)
    assert abs(st["dual_obj"] - ref.dual_obj) <= W_RTOL * abs(ref.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= C0.C) and abs(a @ y) <= 1e-9 * C0.C * len(y)
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, C0.gamma, dev(Xt)).cpu().numpy()
    d_ref = oracle.decision(X, y, ref.alpha, ref.b, Xt, C0.gamma)
    check_decisions(d_gpu, d_ref)


@pytest.mark.parametrize("steps", [1, 10, 100, 1000])
def test_gradient_snapshots_c0(c0, steps):
    X, y, _, _ = c0
    r = oracle.train(X, y, C0.C, C0.gamma, C0.tol, max_iter=steps, want_f=True)
    for gram in (svmx.GRAM_ON, svmx.GRAM_OFF):
        f = torch.empty(X.shape[0], dtype=torch.float64, device="cuda")
        out = svmx.svm_train(dev(X), dev(y), C0.C, C0.gamma, C0.tol, gram=gram, max_iter=steps, f_out=f)
        expect = svmx.SVM_OK if r.status == 0 else svmx.SVM_NOT_CONVERGED
        assert out.status == expect
        assert np.max(np.abs(f.cpu().numpy() - r.f)) <= F_ATOL
        np.testing.assert_allclose(out.alpha.cpu().numpy(), r.alpha, atol=1e-5, rtol=0)


# --- edge cases --------------------------------------------------------------------------

def test_two_point_rbf_gpu():
    X = np.array([[1.0, 2.0, 0.5], [-0.5, 1.0, 2.0]], np.float32)
    y = np.array([1, -1], np.int32)
    for C_, a_exp in ((10.0, 1.2377002127605519), (0.5, 0.5)):
        out = svmx.svm_train(dev(X), dev(y), C_, 0.3, 1e-9)
        assert out.stats["iterations"] == 1
        np.testing.assert_allclose(out.alpha.cpu().numpy(), [a_exp, a_exp], rtol=1e-6)
        assert abs(out.b) <= 1e-7


@pytest.mark.parametrize("n,wgs,gram", [(3, 0, 1), (255, 0, 1), (257, 2, 1), (1001, 5, 2), (4097, 0, 1), (5000, 0, 1),
                                        (5000, 0, 2), (6001, 13, 1)])
def test_ragged_sizes(n, wgs, gram):
    X, y = synth.two_blobs(n, 6, seed=n)
    if n == 3:
        y = np.array([1, -1, 1], np.int32)
    r = oracle.train(X, y, 1.0, 0.3, 1e-3, trace_len=100)
    out = svmx.svm_train(dev(X), dev(y), 1.0, 0.3, 1e-3, gram=gram, workgroups=wgs, trace_len=100)
    k = min(100, r.iterations + 1)
    np.testing.assert_array_equal(out.trace_ul[:k], r.trace_ul[:k])
    assert abs(out.stats["dual_obj"] - r.dual_obj) <= W_RTOL * abs(r.dual_obj)
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, 0.3, dev(X[:500])).cpu().numpy()
    check_decisions(d_gpu, oracle.decision(X, y, r.alpha, r.b, X[:500], 0.3))


@pytest.mark.parametrize("gram", [svmx.GRAM_ON, svmx.GRAM_OFF])
def test_exchange_configurations_agree(gram):
    """The exchange is an exact reduction under a total order, so the number of workgroups,
    the number of polling waves (one per 64 records) and the number of levels change nothing."""
    X, y = synth.two_blobs(12000, 8, seed=7)
    Xd, yd = dev(X), dev(y)
    kw = dict(gram=gram, max_iter=300, trace_len=300)
    base = svmx.svm_train(Xd, yd, 1.0, 0.3, 1e-3, workgroups=40, exchange_levels=1, **kw)
    for wgs, lv in [(100, 1), (100, 2), (190, 1), (190, 2)]:
        out = svmx.svm_train(Xd, yd, 1.0, 0.3, 1e-3, workgroups=wgs, exchange_levels=lv, **kw)
        assert out.stats["iterations"] == base.stats["iterations"]
        np.testing.assert_array_equal(out.trace_ul, base.trace_ul)
        np.testing.assert_array_equal(out.trace_b, base.trace_b)
        np.testing.assert_array_equal(out.alpha.cpu().numpy(), base.alpha.cpu().numpy())


def test_duplicate_samples_eta_floor():
    X, y = synth.two_blobs(200, 4, seed=1)
    X = np.concatenate([X, X[:20]])
    y = np.concatenate([y, -y[:20]])  # identical points with opposite labels: eta = 0
    r = oracle.train(X, y, 1.0, 0.5, 1e-3)
    out = svmx.svm_train(dev(X), dev(y), 1.0, 0.5, 1e-3)
    assert abs(out.stats["dual_obj"] - r.dual_obj) <= W_RTOL * abs(r.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= 1.0) and abs(a @ y) <= 1e-9 * len(y)


def test_max_iter_not_converged_feasible():
    X, y = synth.two_blobs(500, 5, seed=4)
    out = svmx.svm_train(dev(X), dev(y), 1.0, 0.2, 1e-6, max_iter=7)
    assert out.status == svmx.SVM_NOT_CONVERGED
    assert out.stats["iterations"] == 7
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= 1.0) and abs(a @ y) <= 1e-12 * len(y)
    r = oracle.train(X, y, 1.0, 0.2, 1e-6, max_iter=7)
    assert abs(out.b - r.b) <= F_ATOL


@pytest.mark.parametrize("n,d,gram,steps", [(3000, 8, svmx.GRAM_AUTO, 0), (3000, 8, svmx.GRAM_OFF, 0),
                                           (600_000, 16, svmx.GRAM_OFF, 60)])
def test_results_independent_of_check_cadence(n, d, gram, steps):
    """The same steps, multipliers and bias whether the solve runs in launches of 1, 7, 256 or
    the default number of steps: on the Gram path, on the row path (its resident rows of X are
    loaded into LDS again at every launch) and on the row path with 8 samples a thread (60
    steps)."""
    X, y = synth.two_blobs(n, d, seed=8)
    kw = dict(gram=gram, max_iter=steps) if steps else dict(gram=gram)
    ref = svmx.svm_train(dev(X), dev(y), 1.0, 0.1, 1e-3, **kw)
    assert ref.stats["gram_used"] == (1 if gram == svmx.GRAM_AUTO else 0)
    for ce in (1, 7, 256):
        out = svmx.svm_train(dev(X), dev(y), 1.0, 0.1, 1e-3, check_every=ce, **kw)
        assert torch.equal(out.alpha, ref.alpha) and out.b == ref.b
        assert out.stats["iterations"] == ref.stats["iterations"]
        assert out.stats["launches"] >= ref.stats["iterations"] // ce


def test_row_cache_does_not_change_results():
    X, y = synth.two_blobs(3000, 8, seed=9)
    ld = 3008
    base = svmx.svm_train(dev(X), dev(y), 1.0, 0.1, 1e-3, gram=svmx.GRAM_OFF)
    for slots in (1, 3, 64, 3000):
        out = svmx.svm_train(dev(X), dev(y), 1.0, 0.1, 1e-3, gram=svmx.GRAM_OFF, row_cache_bytes=slots * 4 * ld)
        assert torch.equal(out.alpha, base.alpha) and out.b == base.b


def test_predict_edge_cases():
    X, y = synth.two_blobs(300, 5, seed=21)
    a = np.zeros(300)
    d = svmx.svm_predict(dev(X), dev(y), dev(a), 0.25, 0.3, dev(X[:50])).cpu().numpy()
    assert np.all(d == -0.25)  # no support vector: d = -b
    assert svmx.svm_predict(dev(X), dev(y), dev(a), 0.25, 0.3, dev(X[:0])).numel() == 0
    r = oracle.train(X, y, 1.0, 0.3, 1e-3)
    d1 = svmx.svm_predict(dev(X), dev(y), dev(r.alpha), r.b, 0.3, dev(X[:1])).cpu().numpy()
    assert abs(d1[0] - oracle.decision(X, y, r.alpha, r.b, X[:1], 0.3)[0]) <= PRED_ATOL


def test_deterministic_repeat():
    X, y = synth.two_blobs(4000, 8, seed=12)
    a = svmx.svm_train(dev(X), dev(y), 1.0, 0.1, 1e-3)
    b = svmx.svm_train(dev(X), dev(y), 1.0, 0.1, 1e-3)
    assert torch.equal(a.alpha, b.alpha) and a.b == b.b


# --- predict ----------------------------------------------------------------------------------

@pytest.mark.parametrize("mfma", MFMAS)
@pytest.mark.parametrize("cid,n,m,d", [(0, 1500, 777, 16), (2, 1500, 777, 128), (1, 700, 300, 784), (0, 300, 129, 13)])
def test_predict_matches_oracle_given_alpha(cid, n, m, d, mfma):
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid, n=n, m=m, d=d)
    r = oracle.train(X, y, wl.C, wl.gamma, wl.tol)
    d_ref = oracle.decision(X, y, r.alpha, r.b, Xt, wl.gamma)
    d_gpu = svmx.svm_predict(dev(X), dev(y), dev(r.alpha), r.b, wl.gamma, dev(Xt), gram_mfma=mfma).cpu().numpy()
    # same alpha and b: the only difference is the fp32 kernel values of the MFMA path
    assert np.max(np.abs(d_gpu - d_ref)) <= PRED_ATOL


# --- one-vs-one ---------------------------------------------------------------------------------

def kkt_ok(X, y, a, b, C_, gamma, tol, slack=1e-4):
    """tol-KKT of (a, b) checked in fp64 from scratch (validity when trajectories may differ)."""
    from scipy.spatial.distance import cdist
    K = np.exp(-gamma * cdist(X.astype(np.float64), X.astype(np.float64), "sqeuclidean"))
    f = K @ (a * y) - y
    up = ((y > 0) & (a < C_)) | ((y < 0) & (a > 0))
    low = ((y > 0) & (a > 0)) | ((y < 0) & (a < C_))
    feas = np.all(a >= 0) and np.all(a <= C_) and abs(a @ y) <= 1e-9 * C_ * len(y)
    return feas and np.all(f[up] >= b - tol / 2 - slack) and np.all(f[low] <= b + tol / 2 + slack)


@pytest.mark.parametrize("gram", [svmx.GRAM_ON, svmx.GRAM_OFF])
def test_ovo_pairs_equal_standalone_binary_solves(gram):
    """Every pair of the batched one-launch solve is bit-identical to a binary solve of that pair."""
    k = 4
    X, lab, _, _ = synth.generate(4, n=800, m=1, d=24, classes=k)
    out = svmx.svm_train_ovo(dev(X), dev(lab), k, 10.0, 0.05, 1e-3, gram=gram)
    offs, sizes = svmx.ovo_offsets(lab, k)
    for p, (a, b) in enumerate(oracle.ovo_pairs(k)):
        idx, y = oracle.ovo_local(lab, a, b)
        r = svmx.svm_train(dev(X[idx]), dev(y), 10.0, 0.05, 1e-3, gram=gram)
        assert torch.equal(out.alpha[offs[p]:offs[p] + sizes[p]], r.alpha)
        assert out.b[p] == r.b
        assert out.stats[p]["iterations"] == r.stats["iterations"]


@pytest.mark.parametrize("gram", [svmx.GRAM_ON, svmx.GRAM_OFF])
def test_ovo_small(gram):
    """Against the oracle.  The SMO step leaves f_u = f_l in exact arithmetic, so later
    selections can tie exactly and fp32 kernel values may break such ties the other way; what
    is unique is the optimum, so both sides solve to tol 1e-5 and W, tol-KKT validity,
    decisions and labels are compared."""
    k, tol = 4, 1e-5
    X, lab, Xt, _ = synth.generate(4, n=600, m=300, d=20, classes=k)
    models = oracle.train_ovo(X, lab, k, 10.0, 0.05, tol)
    out = svmx.svm_train_ovo(dev(X), dev(lab), k, 10.0, 0.05, tol, gram=gram)
    assert out.status == svmx.SVM_OK
    offs, sizes = svmx.ovo_offsets(lab, k)
    a = out.alpha.cpu().numpy()
    for p, (idx, y, r) in enumerate(models):
        assert sizes[p] == len(idx)
        ap = a[offs[p]:offs[p] + sizes[p]]
        assert abs(out.stats[p]["dual_obj"] - r.dual_obj) <= W_RTOL * abs(r.dual_obj)
        assert kkt_ok(X[idx], y, ap, out.b[p], 10.0, 0.05, tol, slack=1e-5)
    dec_ref, pred_ref = oracle.predict_ovo(X, lab, k, models, Xt, 0.05)
    dec, pred = svmx.svm_predict_ovo(dev(X), dev(lab), k, out.alpha, out.b, 0.05, dev(Xt))
    check_ovo(dec.cpu().numpy(), pred.cpu().numpy(), dec_ref, k, pred_ref)


def test_paper_shaped_context_runs():
    """The shapes of the paper's own runs (102 features, 200 per class): binary against the
    oracle's trajectory and result, nine-class one-vs-one (36 pairs) against the oracle's optimum
    (tol 1e-5 on both sides, as for the other one-vs-one comparisons)."""
    ps = synth.PAPER_SHAPE
    X, lab = synth.paper_shaped(200, 2, seed=200)
    y = np.where(lab == 0, 1, -1).astype(np.int32)
    r = oracle.train(X, y, ps["C"], ps["gamma"], ps["tol"], trace_len=1000)
    out = svmx.svm_train(dev(X), dev(y), ps["C"], ps["gamma"], ps["tol"], trace_len=1000)
    tied = np.flatnonzero(np.asarray(r.trace_gap)[1:].min(axis=1) < 1e-6)
    k = min(r.iterations + 1, 1000, int(tied[0]) + 1 if tied.size else 1000)
    np.testing.assert_array_equal(out.trace_ul[:k], r.trace_ul[:k])
    assert abs(out.stats["dual_obj"] - r.dual_obj) <= W_RTOL * abs(r.dual_obj)
    check_decisions(svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, ps["gamma"], dev(X)).cpu().numpy(),
                    oracle.decision(X, y, r.alpha, r.b, X, ps["gamma"]))

    k9, tol = 9, 1e-5
    X, lab = synth.paper_shaped(200, k9, seed=200)
    models = oracle.train_ovo(X, lab, k9, ps["C"], ps["gamma"], tol)
    out = svmx.svm_train_ovo(dev(X), dev(lab), k9, ps["C"], ps["gamma"], tol)
    assert out.status == svmx.SVM_OK
    offs, sizes = svmx.ovo_offsets(lab, k9)
    a = out.alpha.cpu().numpy()
    for p, (idx, yp, rp) in enumerate(models):
        ap = a[offs[p]:offs[p] + sizes[p]]
        assert abs(out.stats[p]["dual_obj"] - rp.dual_obj) <= W_RTOL * abs(rp.dual_obj)
        assert kkt_ok(X[idx], yp, ap, out.b[p], ps["C"], ps["gamma"], tol, slack=1e-5)
    dec_ref, pred_ref = oracle.predict_ovo(X, lab, k9, models, X, ps["gamma"])
    dec, pred = svmx.svm_predict_ovo(dev(X), dev(lab), k9, out.alpha, out.b, ps["gamma"], dev(X))
    check_ovo(dec.cpu().numpy(), pred.cpu().numpy(), dec_ref, k9, pred_ref)


def test_ovo_many_classes_in_batches():
    """64 classes: 2016 pairs.  On the row path the device holds fewer pair workgroups than
    that at once, so the pairs run in consecutive launches; every pair must still equal a
    standalone binary solve of it, bit for bit, and the votes must match the oracle's."""
    k = 64
    X, lab = synth.multiclass_blobs(640, 8, k, seed=3)
    out = svmx.svm_train_ovo(dev(X), dev(lab), k, 1.0, 0.5, 1e-3, gram=svmx.GRAM_OFF)
    assert out.status == svmx.SVM_OK
    assert out.stats[0]["launches"] > 1  # batched
    offs, sizes = svmx.ovo_offsets(lab, k)
    pairs = oracle.ovo_pairs(k)
    for p in (0, 1, 255, 256, 1000, len(pairs) - 1):
        a, b = pairs[p]
        idx, y = oracle.ovo_local(lab, a, b)
        r = svmx.svm_train(dev(X[idx]), dev(y), 1.0, 0.5, 1e-3, gram=svmx.GRAM_OFF)
        assert torch.equal(out.alpha[offs[p]:offs[p] + sizes[p]], r.alpha), f"pair {p}"
        assert out.b[p] == r.b
    models = oracle.train_ovo(X, lab, k, 1.0, 0.5, 1e-5)
    dec_ref, pred_ref = oracle.predict_ovo(X, lab, k, models, X, 0.5)
    out5 = svmx.svm_train_ovo(dev(X), dev(lab), k, 1.0, 0.5, 1e-5, gram=svmx.GRAM_OFF)
    dec, pred = svmx.svm_predict_ovo(dev(X), dev(lab), k, out5.alpha, out5.b, 0.5, dev(X))
    check_ovo(dec.cpu().numpy(), pred.cpu().numpy(), dec_ref, k, pred_ref)


def test_ovo_predict_matches_oracle_given_alpha():
    k = 5
    X, lab, Xt, _ = synth.generate(4, n=500, m=200, d=12, classes=k)
    models = oracle.train_ovo(X, lab, k, 1.0, 0.1, 1e-3)
    alpha = np.concatenate([r.alpha for (_, _, r) in models])
    b = np.array([r.b for (_, _, r) in models])
    dec_ref, pred_ref = oracle.predict_ovo(X, lab, k, models, Xt, 0.1)
    dec, pred = svmx.svm_predict_ovo(dev(X), dev(lab), k, dev(alpha), b, 0.1, dev(Xt))
    check_ovo(dec.cpu().numpy(), pred.cpu().numpy(), dec_ref, k, pred_ref, gate=PRED_ATOL)


@pytest.mark.parametrize("k", [5, 12])
@pytest.mark.parametrize("mfma", [svmx.MFMA_SPLIT_F16, svmx.MFMA_F32])
def test_ovo_predict_pairs_equal_binary_predict(k, mfma):
    """One-vs-one prediction runs the pairs together (up to 64 per launch; 12 classes give 66
    pairs, so two launches of each stage), but every pair keeps its own support vectors, split
    count and summation order: its decision values are those of svm_predict on that pair's
    samples alone, bit for bit."""
    X, lab, Xt, _ = synth.generate(4, n=60 * k, m=300, d=20, classes=k)
    out = svmx.svm_train_ovo(dev(X), dev(lab), k, 10.0, 0.05, 1e-3)
    assert out.status == svmx.SVM_OK
    dec, _ = svmx.svm_predict_ovo(dev(X), dev(lab), k, out.alpha, out.b, 0.05, dev(Xt), gram_mfma=mfma)
    offs, sizes = svmx.ovo_offsets(lab, k)
    for p, (a, b) in enumerate(oracle.ovo_pairs(k)):
        idx, y = oracle.ovo_local(lab, a, b)
        d1 = svmx.svm_predict(dev(X[idx]), dev(y), out.alpha[offs[p]:offs[p] + sizes[p]].contiguous(), float(out.b[p]),
                              0.05, dev(Xt), gram_mfma=mfma)
        assert torch.equal(dec[:, p].contiguous(), d1), f"pair {p} ({a}, {b})"


@pytest.mark.parametrize("n,d,res", [(3000, 784, 0), (3000, 784, -1), (3000, 784, 7), (2000, 16, 0), (2000, 100, 0),
                                     (2000, 301, 0), (1500, 1500, 0), (1500, 1500, 3), (700, 4100, 0),
                                     (700, 4100, -1), (600, 3001, 0), (600_000, 16, 0), (600_000, 16, -1),
                                     (600_000, 64, 0), (540_000, 200, 0), (540_000, 33, 0)])
def test_row_path_step_uses_the_kernel_row_values(n, d, res):
    """After one row-path step f equals -y + (c_u K(u, .) + c_l K(l, .)) evaluated on the host from
    svm_kernel_rows' fp32 values, bit for bit, at every sample: the solver's row values are the
    entry point's whether its rows of X sit in LDS (all of them, some, or none) or stream from
    HBM, for lane groups of 64 (784 features), 32 (100), 16 (200), 4 (64) and 1 (16), scalar lanes
    (33, 301, 3001), rows longer than one register block (301, 1500, and 4100 and 3001 with 7 and
    11 later blocks), and with 8 samples a thread (more than 524,288 samples), where rows of up
    to 128 features go in batches of one sample and wider ones in batches of two."""
    X, y = synth.two_blobs(n, d, seed=d + 1)
    Xd, yd = dev(X), dev(y)
    gamma = 1.0 / d
    f = torch.empty(n, dtype=torch.float64, device="cuda")
    out = svmx.svm_train(Xd, yd, 1.0, gamma, 1e-3, gram=svmx.GRAM_OFF, max_iter=1, trace_len=1, resident_rows=res,
                         f_out=f)
    assert out.stats["iterations"] == 1
    st = out.stats["resident_rows"]
    if res == -1:
        assert st == 0
    elif res > 0:
        assert st == res
    else:
        assert st > 0
    u, l = (int(v) for v in out.trace_ul[0])
    K = svmx.svm_kernel_rows(Xd, gamma, np.array([u, l])).cpu().numpy().astype(np.float64)
    a = out.alpha.cpu().numpy()
    yf = y.astype(np.float64)
    cu, cl = a[u] * yf[u], a[l] * yf[l]
    np.testing.assert_array_equal(f.cpu().numpy(), -yf + (cu * K[0] + cl * K[1]))


def test_resident_rows_do_not_change_results():
    """A row-path training to convergence with every row of X streamed, with some resident in
    LDS and with as many as fit: identical steps, multipliers and bias."""
    X, y = synth.two_blobs(4000, 784, seed=11)
    Xd, yd = dev(X), dev(y)
    runs = [svmx.svm_train(Xd, yd, 1.0, 1.0 / 784, 1e-3, gram=svmx.GRAM_OFF, resident_rows=r) for r in (-1, 9, 0)]
    assert runs[2].stats["resident_rows"] > 9
    for r in runs[1:]:
        assert r.stats["iterations"] == runs[0].stats["iterations"]
        assert torch.equal(r.alpha, runs[0].alpha)
        assert r.b == runs[0].b


def test_row_path_beyond_one_launch_is_enomem():
    """A row-path problem needing more solver workgroups than the device holds at once (256 of
    4,096 samples) is refused on the host before the cooperative launch, with SVM_ENOMEM."""
    n, d = 1_100_000, 4
    X = torch.rand(n, d, device="cuda")
    y = torch.where(torch.arange(n, device="cuda") % 2 == 0, 1, -1).to(torch.int32)
    with pytest.raises(svmx.SvmError) as e:
        svmx.svm_train(X, y, 1.0, 0.5, 1e-3, gram=svmx.GRAM_OFF, max_iter=10)
    assert e.value.status == svmx.SVM_ENOMEM
    assert "do not fit" in str(e.value)


@pytest.mark.parametrize("gram", [svmx.GRAM_ON, svmx.GRAM_OFF])
@pytest.mark.parametrize("C_,gamma", [(1e-3, 0.125), (1e3, 0.125), (1.0, 10.0)])
def test_extreme_box_and_width(C_, gamma, gram):
    """Degenerate regimes of the dual: C = 1e-3 (most multipliers end at the bound C), C = 1e3
    (near hard margin, large multipliers), gamma = 10 (K close to the identity: every sample a
    support vector).  Against the oracle: the selections up to the first near-tie (early in the
    first and last regimes, where the steps leave exact ties), W, the box and equality
    constraints, tol-KKT with f recomputed by the oracle from the GPU's alpha, and the
    decisions within 1e-3 (measured on MI355X: 4.4e-4 at C = 1e3, where sum a = 2,767, about
    1e-8 in the other two regimes)."""
    X, y = synth.two_blobs(600, 8, seed=17)
    Xt, _ = synth.two_blobs(200, 8, seed=18)
    tol = 1e-3
    r = oracle.train(X, y, C_, gamma, tol, trace_len=500)
    out = svmx.svm_train(dev(X), dev(y), C_, gamma, tol, gram=gram, trace_len=500)
    assert out.status == svmx.SVM_OK
    tied = np.flatnonzero(np.asarray(r.trace_gap)[1:].min(axis=1) < 1e-6)
    k = min(500, r.iterations + 1, out.stats["iterations"] + 1, int(tied[0]) + 1 if tied.size else 500)
    np.testing.assert_array_equal(out.trace_ul[:k], r.trace_ul[:k])
    assert abs(out.stats["dual_obj"] - r.dual_obj) <= W_RTOL * abs(r.dual_obj)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= C_) and abs(a @ y) <= 1e-9 * C_ * len(y)
    f = oracle.f_from_alpha(X, y, a, gamma)
    up = ((y > 0) & (a < C_)) | ((y < 0) & (a > 0))
    low = ((y > 0) & (a > 0)) | ((y < 0) & (a < C_))
    slack = 1e-4 * max(1.0, float(a.sum()))
    assert f[up].min() >= f[low].max() - tol - slack
    d_gpu = svmx.svm_predict(dev(X), dev(y), out.alpha, out.b, gamma, dev(Xt)).cpu().numpy()
    d_ref = oracle.decision(X, y, r.alpha, r.b, Xt, gamma)
    gate = DEC_ATOL
    print(f"\nC={C_} gamma={gamma}: steps {out.stats['iterations']} / {r.iterations}, max |dd| = "
          f"{np.max(np.abs(d_gpu - d_ref)):.2e}, W rel {abs(out.stats['dual_obj'] - r.dual_obj) / abs(r.dual_obj):.1e}, "
          f"trace prefix {k}")
    check_decisions(d_gpu, d_ref, gate)


@pytest.mark.parametrize("bad", [float("nan"), float("inf"), -float("inf")])
def test_non_finite_x_is_rejected(bad):
    """A NaN or an infinity in X would keep every stop test false until max_iter; training
    refuses it up front with SVM_EINVAL (binary, either path, and one-vs-one)."""
    X, y = synth.two_blobs(300, 6, seed=2)
    X[123, 4] = bad
    for gram in (svmx.GRAM_ON, svmx.GRAM_OFF):
        with pytest.raises(svmx.SvmError) as e:
            svmx.svm_train(dev(X), dev(y), 1.0, 0.5, 1e-3, gram=gram)
        assert e.value.status == svmx.SVM_EINVAL and "not finite" in str(e.value)
    lab = (y > 0).astype(np.int32)
    with pytest.raises(svmx.SvmError) as e:
        svmx.svm_train_ovo(dev(X), dev(lab), 2, 1.0, 0.5, 1e-3)
    assert e.value.status == svmx.SVM_EINVAL and "not finite" in str(e.value)
