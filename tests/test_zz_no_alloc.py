"""svm_train_static -- the training entry point that allocates nothing -- against svm_train.

Both run the same kernels on the same plan; svm_train_static takes its device scratch from the
library's static array instead of a caller workspace.  Every case runs two calls in a row on the
static scratch (the second with a smaller input, so stale contents of the first are in the
array) and requires the multipliers, bias, step count, trace and objective of svm_train with the
same options bit for bit.  Sizes beyond the scratch are refused with SVM_EWORKSPACE.
"""
import numpy as np
import pytest
import torch

from paper_2311_14908_amd import svmx, synth

pytestmark = pytest.mark.gpu


def _inputs(cid, n):
    wl = synth.workload(cid)
    X, y, _, _ = synth.generate(cid, n=n, m=1)
    return wl, torch.from_numpy(X).cuda(), torch.from_numpy(y).cuda()


def _same(ref, got):
    assert got.status == ref.status
    assert torch.equal(got.alpha, ref.alpha)
    assert got.b == ref.b
    for k in ("iterations", "n_sv", "n_bound_sv", "b_up", "b_low", "dual_obj", "gram_used", "launches"):
        assert got.stats[k] == ref.stats[k], k
    assert np.array_equal(got.trace_ul, ref.trace_ul)
    assert np.array_equal(got.trace_b, ref.trace_b, equal_nan=True)


@pytest.mark.parametrize("cid,sizes,opt_ref,opt_static", [
    # Gram path (the Gram fits the scratch)
    (0, (3000, 1200), dict(gram=svmx.GRAM_ON), dict()),
    # row path, 784 features
    (1, (20000, 5000), dict(gram=svmx.GRAM_OFF), dict(gram=svmx.GRAM_OFF)),
    # AUTO without room for the Gram falls back to the row path; then a size whose Gram fits
    (3, (6000, 2500), dict(gram=svmx.GRAM_OFF), dict()),
])
def test_static_matches_workspace_entry(gpu_ok, cid, sizes, opt_ref, opt_static):
    for k, n in enumerate(sizes):
        wl, Xd, yd = _inputs(cid, n)
        o_ref = dict(opt_ref)
        if cid == 3 and k == 1:
            o_ref = dict(gram=svmx.GRAM_ON)  # 2,500 samples: the static plan takes the Gram too
        ref = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, trace_len=300, **o_ref)
        alpha = torch.empty(n, dtype=torch.float64, device="cuda")
        torch.cuda.synchronize()
        got = svmx.svm_train_static(Xd, yd, wl.C, wl.gamma, wl.tol, alpha=alpha, trace_len=300, **opt_static)
        print(f"static: workload {cid} n={n} gram_used={got.stats['gram_used']} steps={got.stats['iterations']}",
              flush=True)
        _same(ref, got)
        assert got.alpha.data_ptr() == alpha.data_ptr()


def test_static_refuses_plans_beyond_the_scratch(gpu_ok):
    wl, Xd, yd = _inputs(0, 5000)
    with pytest.raises(svmx.SvmError) as e:
        svmx.svm_train_static(Xd, yd, wl.C, wl.gamma, wl.tol, gram=svmx.GRAM_ON)
    assert e.value.status == svmx.SVM_EWORKSPACE
    assert "svm_train_static" in str(e.value)
    # the array is still usable afterwards
    wl, Xd, yd = _inputs(0, 800)
    ref = svmx.svm_train(Xd, yd, wl.C, wl.gamma, wl.tol, trace_len=50)
    got = svmx.svm_train_static(Xd, yd, wl.C, wl.gamma, wl.tol, trace_len=50)
    _same(ref, got)
