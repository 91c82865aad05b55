"""One launch per outer iteration (svm_params.fused) against the two-launch
loop (selection, then row update).

Every block of the one-launch kernel merges the previous launch's candidate
records, solves the same subproblem and updates its rows; the selection is
exact and the kernel values, the update order and the subproblem are the
two-launch loop's, so a training must give the same alpha, iterations,
bias and objective bit for bit.  Shapes cover working sets of 2, 6 and 16,
ragged row and feature tails, several feature slabs, eps-SVR, every kernel
function, held-out folds (cross-validation), one-vs-rest and tiny n.
"""
import numpy as np
import pytest

from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _both(X, y, **kw):
    out = []
    for fused in (0, 1):
        m = nv.svm_train(X, y, cache_bytes=-1, fused=fused, **kw)
        idx, coef, alpha = nv.svm_model_get(m, 0, with_alpha=True)
        out.append((m.info(), alpha))
    return out


def _same(two, one):
    (i2, a2), (i1, a1) = two, one
    np.testing.assert_array_equal(a1, a2)
    for k in ("iters", "b", "dual_obj", "kernel_rows", "gap", "n_sv_output"):
        assert i1[k] == i2[k], (k, i1[k], i2[k])


CASES = [  # name, n, d (None: the workload's), q, extra params
    ("C1", 2000, None, 16, {}),
    ("C1", 2000, None, 6, {}),
    ("C1", 1500, None, 2, {}),
    ("C2", 3000, None, 16, {}),
    ("C3", 6000, None, 16, {}),
    ("C3", 100, None, 16, {}),
    ("C3", 5000, 7, 16, {}),
    ("C3", 3000, 300, 16, {}),
    ("C1", 2000, None, 16, {"kernel": nv.SVM_KERNEL_POLY, "coef0": 1.0,
                            "tol": 1e-2}),
    ("C1", 2000, None, 16, {"kernel": nv.SVM_KERNEL_SIGMOID}),
    ("C1", 2000, None, 16, {"kernel": nv.SVM_KERNEL_LINEAR, "tol": 1e-2}),
]


@pytest.mark.parametrize("name,n,d,q,extra", CASES)
def test_one_launch_matches_two_launches(name, n, d, q, extra):
    w = workloads.make(name, n=n, n_test=10)
    X = w.X if d is None else np.ascontiguousarray(w.X[:, :d])
    gamma = w.gamma if d is None else 1.0 / d
    kw = dict(type=w.type, C=w.C, epsilon=w.eps, gamma=gamma, tol=w.tol,
              working_set=q)
    kw.update(extra)
    two, one = _both(X, w.y, **kw)
    assert one[0]["status"] == nv.SVM_OK
    _same(two, one)


def test_one_launch_cross_validation():
    w = workloads.c1(n=1800, n_test=10)
    res = []
    for fused in (0, 1):
        D, st = nv.svm_cross_validate(w.X, w.y, k=5, C=w.C, gamma=w.gamma,
                                      tol=w.tol, cache_bytes=-1, fused=fused)
        res.append((D, st))
    np.testing.assert_array_equal(res[0][0], res[1][0])
    assert res[0][1]["iters"] == res[1][1]["iters"]


def test_one_launch_ovr():
    w = workloads.make("C4", n=3000, n_test=10)
    ms = [nv.svm_train_ovr(w.X, w.y, w.n_classes, C=w.C, gamma=w.gamma,
                           tol=w.tol, cache_bytes=-1, fused=f)
          for f in (0, 1)]
    for c in range(w.n_classes):
        a0 = nv.svm_model_get(ms[0], c, with_alpha=True)[2]
        a1 = nv.svm_model_get(ms[1], c, with_alpha=True)[2]
        np.testing.assert_array_equal(a0, a1)
        assert ms[0].info(c)["iters"] == ms[1].info(c)["iters"]
