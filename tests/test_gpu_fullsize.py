"""GPU vs oracle at the full sizes of the synthetic workloads, through the C ABI.

The oracle's full-size results are stored in tests/golden/oracle_full_w*.json, written by
tests/golden/make_oracle_refs.py (which calls only oracle/).  The inputs are regenerated here
and their digest must equal the one stored with the reference.

Gates (as for the small cases):
  working set   identical (u, l) for the first 1000 steps, up to the first step whose oracle
                runner-up gap is below 1e-6 (a tie within the fp32-kernel error of f, where
                either choice is a maximal violating pair)
  objective     relative 1e-4
  decisions     max abs 1e-3 on the stored test points; labels compared on every point (one-vs-one:
                the voted class must be one the oracle's decisions allow, exactly the oracle's
                where no pair decision is within the measured error of zero)
  validity      0 <= a <= C, sum a y = 0, tol-KKT on every row with f recomputed by the oracle
                from the GPU's alpha (slack 1e-4 for the fp32 kernel values), and the duality
                gap 0 <= P - W <= n C tol from the same f
"""
import hashlib
import json
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2311_14908_amd import svmx, synth
from tests.label_checks import check_binary_labels, check_ovo_predictions, kkt_and_gap, ovo_vote

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TIE_GAP = 1e-6


def ref(cid):
    path = os.path.join(GOLDEN, f"oracle_full_w{cid}.json")
    if not os.path.exists(path):
        pytest.skip(f"{path} not generated")
    return json.load(open(path))


def digest(*arrays):
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    svmx.load()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.mark.parametrize("cid,gram", [(1, svmx.GRAM_AUTO), (2, svmx.GRAM_AUTO), (3, svmx.GRAM_AUTO),
                                      (1, svmx.GRAM_OFF), (2, svmx.GRAM_OFF), (3, svmx.GRAM_OFF)])
def test_binary_full_size(cid, gram):
    """The default path (the Gram fits at all three sizes) and the row path (rows of X resident
    in LDS as far as they fit: part of each slice at 784 features, all of it at 128 and 32)."""
    R = ref(cid)
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid)
    nt = len(R["test_decisions"])
    assert digest(X, y, Xt[:nt]) == R["inputs_sha256"], "inputs differ from the stored reference"
    Xd, yd = dev(X), dev(y)
    out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, trace_len=1000, gram=gram)
    assert out.status == svmx.SVM_OK
    st = out.stats
    assert st["gram_used"] == (1 if gram == svmx.GRAM_AUTO else 0)
    if gram == svmx.GRAM_OFF:
        assert st["resident_rows"] > 0
    print(f"\nworkload {cid}: gpu {st['iterations']} steps W={st['dual_obj']:.9f} b={out.b:.6f}; "
          f"oracle {R['iterations']} steps W={R['dual_obj']:.9f} b={R['b']:.6f}")

    # working-set sequence
    gaps = np.array(R["trace_gap_min"])
    tied = np.flatnonzero(gaps[1:] < TIE_GAP)
    k = min(len(R["trace_ul"]), 1000, (int(tied[0]) + 1) if tied.size else 1000)
    np.testing.assert_array_equal(out.trace_ul[:k], np.array(R["trace_ul"])[:k])

    # objective and decisions
    assert abs(st["dual_obj"] - R["dual_obj"]) <= 1e-4 * abs(R["dual_obj"])
    d_gpu = svmx.svm_predict(Xd, yd, out.alpha, out.b, wl.gamma, dev(Xt[:nt])).cpu().numpy()
    d_ref = np.array(R["test_decisions"])
    err = float(np.max(np.abs(d_gpu - d_ref)))
    print(f"max |d_gpu - d_oracle| = {err:.2e}")
    assert err <= 1e-3
    check_binary_labels(d_gpu, d_ref, err)

    # validity of the GPU solution, checked by the oracle on every row
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= wl.C)
    assert abs(float(a @ y)) <= 1e-9 * wl.C * len(y)
    f = oracle.f_from_alpha(X, y, a, wl.gamma)
    gap, _ = kkt_and_gap(f, y, a, out.b, wl.C, wl.tol, slack=1e-4)
    print(f"duality gap P - W = {gap:.3e} (bound n C tol = {len(y) * wl.C * wl.tol:.1f})")


@pytest.mark.parametrize("gram", [svmx.GRAM_AUTO, svmx.GRAM_OFF])
def test_ovo_full_size(gram):
    """All 45 pairs of the 60,000 x 784 workload to convergence, from the class-sorted global Gram
    (default) or on the row path: every pair's W against the stored oracle optimum, decisions and
    votes on the stored test points."""
    R = ref(4)
    wl = synth.workload(4)
    k = wl.classes
    X, lab, Xt, _ = synth.generate(4)
    nt = len(R["test_pred"])
    assert digest(X, lab, Xt[:nt]) == R["inputs_sha256"], "inputs differ from the stored reference"
    Xd, ld = dev(X), dev(lab)
    out = svmx.svm_train_ovo(Xd, ld, k, wl.C, wl.gamma, wl.tol, gram=gram)
    assert out.status == svmx.SVM_OK
    assert all(st["gram_used"] == (1 if gram == svmx.GRAM_AUTO else 0) for st in out.stats)
    for p, rp in enumerate(R["pairs"]):
        assert abs(out.stats[p]["dual_obj"] - rp["dual_obj"]) <= 1e-4 * abs(rp["dual_obj"])
    dec, pred = svmx.svm_predict_ovo(Xd, ld, k, out.alpha, out.b, wl.gamma, dev(Xt[:nt]))
    d_ref = np.array(R["test_decisions"])
    dec = dec.cpu().numpy()
    err = float(np.max(np.abs(dec - d_ref)))
    print(f"\none-vs-one (gram {gram}): max |d_gpu - d_oracle| = {err:.2e}")
    assert err <= 1e-3
    # the vote restated in the checks gives the oracle's stored classes from its stored decisions
    assert [ovo_vote(r > 0, k) for r in d_ref] == list(R["test_pred"])
    check_ovo_predictions(pred.cpu().numpy(), d_ref, k, err)


def test_ovo_row_path_full_size_pairs_equal_binary():
    """One-vs-one on the row path at the full workload size (45 pairs of 12000 samples in one
    cooperative launch, the workgroup budget fitted to what the device holds at once): after a
    fixed number of steps every pair equals a standalone binary row-path solve of that pair,
    bit for bit (the row values of a sample do not depend on how samples are spread over
    workgroups, and the exchange is an exact reduction)."""
    wl = synth.workload(4)
    k = wl.classes
    X, lab, _, _ = synth.generate(4, m=1)
    steps = 200
    Xd, ld = dev(X), dev(lab)
    out = svmx.svm_train_ovo(Xd, ld, k, wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_OFF, max_iter=steps)
    assert out.status in (svmx.SVM_OK, svmx.SVM_NOT_CONVERGED)
    offs, sizes = svmx.ovo_offsets(lab, k)
    for p, (a, b) in enumerate(oracle.ovo_pairs(k)):
        idx, y = oracle.ovo_local(lab, a, b)
        r = svmx.svm_train(dev(X[idx]), dev(y), wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_OFF, max_iter=steps)
        assert out.stats[p]["iterations"] == r.stats["iterations"]
        assert torch.equal(out.alpha[offs[p]:offs[p] + sizes[p]], r.alpha), f"pair {p}"


@pytest.mark.parametrize("cid,q,gram", [(1, 128, svmx.GRAM_AUTO), (1, 128, svmx.GRAM_OFF), (2, 32, svmx.GRAM_AUTO),
                                        (2, 32, svmx.GRAM_OFF), (3, 32, svmx.GRAM_AUTO), (3, 32, svmx.GRAM_OFF)])
def test_working_set_full_size(cid, q, gram):
    """The working-set solver at the full sizes reaches the optimum of the stored oracle
    solve (its trajectory differs from the pair steps', so the gates are those of the optimum):
    W within 1e-4, the stored test decisions within 1e-3 with their labels, the box and
    equality constraints, and tol-KKT on 128 rows whose f the oracle recomputes."""
    R = ref(cid)
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid)
    nt = len(R["test_decisions"])
    assert digest(X, y, Xt[:nt]) == R["inputs_sha256"], "inputs differ from the stored reference"
    Xd, yd = dev(X), dev(y)
    out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, working_set=q, gram=gram)
    assert out.status == svmx.SVM_OK
    st = out.stats
    print(f"\nworkload {cid}, q={q}, gram_used={st['gram_used']}: {st['rounds']} rounds, {st['iterations']} pair "
          f"steps, W={st['dual_obj']:.9f} (oracle {R['dual_obj']:.9f})")
    assert abs(st["dual_obj"] - R["dual_obj"]) <= 1e-4 * abs(R["dual_obj"])
    d_gpu = svmx.svm_predict(Xd, yd, out.alpha, out.b, wl.gamma, dev(Xt[:nt])).cpu().numpy()
    d_ref = np.array(R["test_decisions"])
    err = float(np.max(np.abs(d_gpu - d_ref)))
    assert err <= 1e-3
    check_binary_labels(d_gpu, d_ref, err)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= wl.C)
    assert abs(float(a @ y)) <= 1e-9 * wl.C * len(y)
    f = oracle.f_from_alpha(X, y, a, wl.gamma)
    kkt_and_gap(f, y, a, out.b, wl.C, wl.tol, slack=1e-4)


@pytest.mark.parametrize("cid,gram,schedule", [(1, svmx.GRAM_AUTO, 1), (2, svmx.GRAM_AUTO, 1), (3, svmx.GRAM_AUTO, 1),
                                               (1, svmx.GRAM_OFF, 1), (3, svmx.GRAM_OFF, None)])
def test_auto_full_size(cid, gram, schedule):
    """working_set = AUTO at the full workload sizes: the schedule its rule picks (rounds on all
    three: on the 8-component mixture the probe's rounds hold about as many pair steps as they
    cost, at the threshold), and the optimum gates against the stored oracle solve: W, decisions
    and labels, tol-KKT and the duality gap on every row."""
    R = ref(cid)
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid)
    nt = len(R["test_decisions"])
    assert digest(X, y, Xt[:nt]) == R["inputs_sha256"], "inputs differ from the stored reference"
    Xd, yd = dev(X), dev(y)
    out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=svmx.WORKING_SET_AUTO)
    assert out.status == svmx.SVM_OK
    st = out.stats
    print(f"\nworkload {cid} gram {gram}: schedule {st['schedule']}, {st['rounds']} rounds, {st['iterations']} pair "
          f"steps, W={st['dual_obj']:.9f} (oracle {R['dual_obj']:.9f})")
    if schedule is not None:
        assert st["schedule"] == schedule
    assert abs(st["dual_obj"] - R["dual_obj"]) <= 1e-4 * abs(R["dual_obj"])
    d_gpu = svmx.svm_predict(Xd, yd, out.alpha, out.b, wl.gamma, dev(Xt[:nt])).cpu().numpy()
    d_ref = np.array(R["test_decisions"])
    err = float(np.max(np.abs(d_gpu - d_ref)))
    assert err <= 1e-3
    check_binary_labels(d_gpu, d_ref, err)
    a = out.alpha.cpu().numpy()
    assert np.all(a >= 0) and np.all(a <= wl.C)
    assert abs(float(a @ y)) <= 1e-9 * wl.C * len(y)
    f = oracle.f_from_alpha(X, y, a, wl.gamma)
    kkt_and_gap(f, y, a, out.b, wl.C, wl.tol, slack=1e-4)


def test_rounds_past_the_lds_rows():
    """140,000 samples of the 100,000 x 32 recipe with the Gram and working_set = AUTO: the 255
    owners hold slices of 549-550 samples, more than the 16,384 / 32 = 512 whose Gram rows of B
    fit in LDS, so every round's f update also reads the rest of each slice from the Gram.  The
    schedule stays on rounds and the solution passes feasibility, tol-KKT and the duality gap on
    every row with f recomputed by the oracle from the GPU's alpha."""
    wl = synth.workload(3)
    n = 140_000
    assert -(-n // 255) > 16_384 // 32
    X, y, _, _ = synth.generate(3, n=n, m=1)
    Xd, yd = dev(X), dev(y)
    out = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_ON, working_set=svmx.WORKING_SET_AUTO)
    assert out.status == svmx.SVM_OK
    st = out.stats
    print(f"\nn={n}: schedule {st['schedule']}, {st['rounds']} rounds, {st['iterations']} pair steps, "
          f"W={st['dual_obj']:.9f}")
    assert st["schedule"] == 1
    a = out.alpha.cpu().numpy()
    b = out.b
    del out, Xd, yd
    torch.cuda.empty_cache()
    assert np.all(a >= 0) and np.all(a <= wl.C)
    assert abs(float(a @ y)) <= 1e-9 * wl.C * n
    f = oracle.f_from_alpha(X, y, a, wl.gamma)
    gap, W = kkt_and_gap(f, y, a, b, wl.C, wl.tol, slack=1e-4)
    assert abs(W - st["dual_obj"]) <= 1e-6 * abs(W)
