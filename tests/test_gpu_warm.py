"""Warm start (a given alpha instead of 0) on the GPU.

A feasible start changes the path, not the optimum: from the converged alpha
of the same problem the solve stops at once with the same objective; from
the solution at a smaller C (feasible for a larger C) it reaches the
oracle's cold-start optimum at the larger C, to the usual bars, in fewer
outer iterations than a cold start.
"""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _alpha(m):
    return nv.svm_model_get(m, 0, with_alpha=True)[2]


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_restart_from_converged_alpha(name):
    w = workloads.make(name, n=2000, n_test=10)
    kw = dict(type=w.type, C=w.C, epsilon=w.eps, gamma=w.gamma, tol=w.tol)
    m = nv.svm_train(w.X, w.y, **kw)
    m2 = nv.svm_train(w.X, w.y, alpha0=_alpha(m), **kw)
    i1, i2 = m.info(), m2.info()
    assert i2["iters"] <= 1
    assert i2["dual_obj"] == pytest.approx(i1["dual_obj"], rel=1e-9)
    assert i2["gap"] <= w.tol


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_warm_start_along_c(name):
    w = workloads.make(name, n=2000, n_test=500)
    kw = dict(type=w.type, epsilon=w.eps, gamma=w.gamma, tol=w.tol)
    C2 = 4.0 * w.C
    m1 = nv.svm_train(w.X, w.y, C=w.C, **kw)
    cold = nv.svm_train(w.X, w.y, C=C2, **kw)
    warm = nv.svm_train(w.X, w.y, C=C2, alpha0=_alpha(m1), **kw)
    p = Params(w.type, C=C2, eps=w.eps, gamma=w.gamma, tol=w.tol)
    ref = oracle.train(w.X, w.y, p)
    iw, ic = warm.info(), cold.info()
    assert iw["status"] == nv.SVM_OK
    assert iw["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)
    assert iw["iters"] < ic["iters"]
    a = _alpha(warm)
    assert np.all(a >= 0) and np.all(a <= C2)
    D = nv.svm_predict(warm, w.Xt)
    Dref = oracle.model_decision(w.X, w.y, p, ref, w.Xt)
    assert np.max(np.abs(D - Dref)) <= 1e-3
