"""Oracle endpoint against scikit-learn's bundled LIBSVM (Chang & Lin 2011).

LIBSVM selects pairs with second-order information (not the maximal
violating pair), so only the endpoint is comparable: dual objective within
1e-4 relative, decision values within the stopping slack at tol 1e-3, and
labels.  Same RBF parameterisation (gamma), no shrinking.
"""
import numpy as np
import pytest
from sklearn.metrics.pairwise import rbf_kernel
from sklearn.svm import SVC, SVR

from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import workloads


def _dual_obj_svc(K, y, coef_full):
    # f = 1/2 c^T K c - sum a,  with c_i = y_i a_i
    return 0.5 * coef_full @ K @ coef_full - np.sum(np.abs(coef_full))


def test_c1_svc_endpoint(orc):
    w = workloads.c1()
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=1e-3)
    r = orc.train(w.X, w.y, p)
    D = orc.model_decision(w.X, w.y, p, r, w.Xt)

    lib = SVC(C=w.C, kernel="rbf", gamma=w.gamma, tol=1e-3, shrinking=False)
    lib.fit(w.X.astype(np.float64), w.y)
    assert list(lib.classes_) == [-1.0, 1.0]
    Dl = lib.decision_function(w.Xt.astype(np.float64))
    cl = np.zeros(w.n)
    cl[lib.support_] = lib.dual_coef_[0]
    K = rbf_kernel(w.X.astype(np.float64), gamma=w.gamma)
    f_lib = _dual_obj_svc(K, w.y, cl)
    assert r.obj == pytest.approx(f_lib, rel=1e-4)
    np.testing.assert_allclose(D, Dl, atol=2e-3)
    agree = np.mean(np.sign(D + 1e-300) == np.sign(Dl + 1e-300))
    assert agree >= 0.999
    # the constant term: LIBSVM's intercept is our b
    assert r.b == pytest.approx(lib.intercept_[0], abs=2e-3)


def test_c2_svr_endpoint(orc):
    w = workloads.c2(n=2000, n_test=1000)
    p = Params(EPS_SVR, C=w.C, eps=w.eps, gamma=w.gamma, tol=1e-3)
    r = orc.train(w.X, w.y, p)
    D = orc.model_decision(w.X, w.y, p, r, w.Xt)

    lib = SVR(C=w.C, epsilon=w.eps, kernel="rbf", gamma=w.gamma, tol=1e-3,
              shrinking=False)
    lib.fit(w.X.astype(np.float64), w.y.astype(np.float64))
    Dl = lib.predict(w.Xt.astype(np.float64))
    cl = np.zeros(w.n)
    cl[lib.support_] = lib.dual_coef_[0]
    c = orc.coefficients(EPS_SVR, w.n, w.y, r.alpha)
    K = rbf_kernel(w.X.astype(np.float64), gamma=w.gamma)
    z = w.y.astype(np.float64)
    f_lib = 0.5 * cl @ K @ cl + w.eps * np.abs(cl).sum() - z @ cl
    f_or = 0.5 * c @ K @ c + w.eps * np.abs(c).sum() - z @ c
    assert r.obj == pytest.approx(f_or, rel=1e-9)
    assert f_or == pytest.approx(f_lib, rel=1e-4)
    np.testing.assert_allclose(D, Dl, atol=2e-3)
