"""Warm start of a binary training (svm_options.alpha_init, f_init) through the C ABI.

- Resumed from the multipliers and the f_out of a training stopped by max_iter, the per-step
  solver takes exactly the steps the uninterrupted training takes: the selections of every later
  step, the final multipliers and b are bit for bit those of one uninterrupted call (Gram path
  with one and with several workgroups, row path).
- Resumed from the multipliers alone, f is recomputed on the device (f_i = sum a_j y_j K_ij - y_i
  over the support vectors): at an optimal start the call takes no step and its f equals the
  incremental f of the training that found it within 1e-9 (Gram path); from a partial start the
  training reaches the same optimum (dual objective within 1e-6 relative, decisions within the
  1e-3 gate of the decision parity tests: on the row path f is recomputed with the exact kernel,
  the steps use fp32 kernel values, so the two stop at different points within tol), with the
  pair steps and with the working-set rounds.
- Starting points that break the box or the equality constraint, f_init without alpha_init, and
  a warm start of a one-vs-one training are refused with SVM_EINVAL.
"""
import numpy as np
import pytest
import torch

from paper_2311_14908_amd import svmx, synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    svmx.load()


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def problem(cid, n):
    wl = synth.workload(cid)
    X, y, Xt, _ = synth.generate(cid, n=n, m=2000)
    return wl, dev(X), dev(y), dev(Xt)


CASES = [(0, None, svmx.GRAM_ON), (3, 20000, svmx.GRAM_ON), (2, 8000, svmx.GRAM_OFF)]


@pytest.mark.parametrize("cid,n,gram", CASES)
def test_resume_with_f_takes_the_same_steps(cid, n, gram):
    wl, Xd, yd, _ = problem(cid, n)
    nn = Xd.shape[0]
    full = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, trace_len=100000)
    steps = full.stats["iterations"]
    k = steps // 3
    assert k > 10
    f_k = torch.empty(nn, dtype=torch.float64, device=Xd.device)
    part = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, max_iter=k, f_out=f_k)
    assert part.status == svmx.SVM_NOT_CONVERGED and part.stats["iterations"] == k
    rest = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, trace_len=100000, alpha_init=part.alpha,
                          f_init=f_k)
    print(f"\nworkload {cid} n={nn} gram={gram}: {steps} steps uninterrupted, {k} + {rest.stats['iterations']} resumed")
    assert rest.status == svmx.SVM_OK
    assert rest.stats["iterations"] == steps - k
    m = min(len(rest.trace_ul), len(full.trace_ul) - k)
    assert m > 0 and np.array_equal(rest.trace_ul[:m], full.trace_ul[k:k + m])
    assert torch.equal(rest.alpha, full.alpha) and rest.b == full.b


def dual(alpha, y, f):
    """W = 1/2 sum a - 1/2 sum a y f (the finalize's dual objective)."""
    a, yy, ff = alpha.cpu().numpy(), y.cpu().numpy().astype(np.float64), f.cpu().numpy()
    return 0.5 * a.sum() - 0.5 * float(np.dot(a * yy, ff))


def test_recomputed_f_at_the_optimum():
    wl, Xd, yd, _ = problem(3, 20000)
    nn = Xd.shape[0]
    f_ref = torch.empty(nn, dtype=torch.float64, device=Xd.device)
    full = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_ON, f_out=f_ref)
    f_re = torch.empty_like(f_ref)
    again = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_ON, alpha_init=full.alpha, f_out=f_re)
    err = float(torch.max(torch.abs(f_re - f_ref)))
    print(f"\nrecomputed f against the incremental f: {err:.2e}")
    assert again.status == svmx.SVM_OK and again.stats["iterations"] == 0
    assert err <= 1e-9
    assert torch.equal(again.alpha, full.alpha)


@pytest.mark.parametrize("cid,n,gram,q", [(3, 20000, svmx.GRAM_ON, 0), (2, 8000, svmx.GRAM_OFF, 0),
                                          (3, 20000, svmx.GRAM_ON, 32), (0, None, svmx.GRAM_OFF, 32)])
def test_resume_from_alpha_reaches_the_optimum(cid, n, gram, q):
    wl, Xd, yd, Td = problem(cid, n)
    nn = Xd.shape[0]
    f_a = torch.empty(nn, dtype=torch.float64, device=Xd.device)
    full = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=q, f_out=f_a)
    k = full.stats["iterations"] // 2
    part = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=q, max_iter=k)
    f_c = torch.empty_like(f_a)
    rest = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, gram=gram, working_set=q, alpha_init=part.alpha, f_out=f_c)
    assert rest.status == svmx.SVM_OK
    wa, wc = dual(full.alpha, yd, f_a), dual(rest.alpha, yd, f_c)
    da = svmx.svm_predict(Xd, yd, full.alpha, full.b, wl.gamma, Td).cpu().numpy()
    dc = svmx.svm_predict(Xd, yd, rest.alpha, rest.b, wl.gamma, Td).cpu().numpy()
    derr = float(np.max(np.abs(da - dc)))
    print(f"\nworkload {cid} n={nn} gram={gram} q={q}: W {wa:.10g} / {wc:.10g}, decisions {derr:.2e}, "
          f"{full.stats['iterations']} steps uninterrupted, {part.stats['iterations']} + {rest.stats['iterations']}")
    assert abs(wc - wa) <= 1e-6 * abs(wa)
    assert derr <= 1e-3


def expect_einval(fn):
    with pytest.raises(svmx.SvmError) as e:
        fn()
    assert e.value.status == svmx.SVM_EINVAL


def test_invalid_starts_are_refused():
    wl, Xd, yd, _ = problem(0, None)
    nn = Xd.shape[0]
    y = yd.cpu().numpy()
    train = lambda **kw: svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, **kw)
    bad = torch.zeros(nn, dtype=torch.float64, device=Xd.device)
    bad[0] = -1e-3
    expect_einval(lambda: train(alpha_init=bad))                       # below the box
    bad = torch.zeros(nn, dtype=torch.float64, device=Xd.device)
    bad[0] = 2 * wl.C
    expect_einval(lambda: train(alpha_init=bad))                       # above the box
    bad = torch.zeros(nn, dtype=torch.float64, device=Xd.device)
    bad[0] = wl.C / 2
    expect_einval(lambda: train(alpha_init=bad))                       # sum a y != 0
    bad[0] = float("nan")
    expect_einval(lambda: train(alpha_init=bad))                       # not finite
    good = torch.zeros(nn, dtype=torch.float64, device=Xd.device)
    i, j = int(np.flatnonzero(y > 0)[0]), int(np.flatnonzero(y < 0)[0])
    good[i] = good[j] = wl.C / 4                                       # feasible
    assert train(alpha_init=good).status == svmx.SVM_OK
    f_bad = torch.full((nn,), float("inf"), dtype=torch.float64, device=Xd.device)
    expect_einval(lambda: train(alpha_init=good, f_init=f_bad))        # f not finite
    expect_einval(lambda: train(f_init=torch.zeros(nn, dtype=torch.float64, device=Xd.device)))
    lab = torch.from_numpy((np.arange(nn) % 3).astype(np.int32)).cuda()
    expect_einval(lambda: svmx.svm_train_ovo(Xd, lab, 3, wl.C, wl.gamma, wl.tol, alpha_init=good))
