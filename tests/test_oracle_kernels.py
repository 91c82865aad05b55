"""Oracle pins for the linear, polynomial and sigmoid kernels.

Section 3 lists four kernel functions (linear, polynomial, radial basis and
sigmoid) without formulas; the oracle takes the e1071/LIBSVM
parameterisation the paper's interface follows:
    linear  u.v,   polynomial (gamma u.v + coef0)^degree,
    sigmoid tanh(gamma u.v + coef0).
Pinned by: scikit-learn's pairwise kernels (dense and CSR input), numbers
worked by hand, the 2-point C-SVC closed form for a general kernel, the
exact QP optimum by active-set enumeration (positive definite cases) and
LIBSVM's endpoint on the same problems.
"""
import numpy as np
import pytest
import scipy.sparse as sp
from sklearn.metrics.pairwise import (linear_kernel, polynomial_kernel,
                                      sigmoid_kernel)
from sklearn.svm import SVC, SVR

from oracle import C_SVC, EPS_SVR, LINEAR, POLY, SIGMOID, Params
from paper_1706_05544_amd import workloads
from paper_1706_05544_amd.workloads import tiny

from test_oracle_bruteforce import brute_force


def _sk_kernel(kind, A, B, gamma, degree, coef0):
    A = A.astype(np.float64)
    B = B.astype(np.float64)
    if kind == LINEAR:
        return linear_kernel(A, B)
    if kind == POLY:
        return polynomial_kernel(A, B, degree=degree, gamma=gamma, coef0=coef0)
    return sigmoid_kernel(A, B, gamma=gamma, coef0=coef0)


KERNELS = [(LINEAR, 0.0, 3, 0.0), (POLY, 0.1, 3, 1.0), (POLY, 0.05, 2, 0.0),
           (POLY, 0.2, 5, -0.5), (SIGMOID, 0.02, 3, 0.0),
           (SIGMOID, 0.1, 3, -1.0)]


@pytest.mark.parametrize("kind,gamma,degree,coef0", KERNELS)
def test_kernel_matches_sklearn(orc, kind, gamma, degree, coef0):
    rng = np.random.default_rng(5)
    A = rng.standard_normal((13, 7)).astype(np.float32)
    B = rng.standard_normal((9, 7)).astype(np.float32)
    B[B < -0.3] = 0.0
    ref = _sk_kernel(kind, A, B, gamma, degree, coef0)
    K = orc.kernel(A, B, gamma, kind, degree, coef0)
    np.testing.assert_allclose(K, ref, rtol=1e-12, atol=1e-13)
    # CSR input (merge over the sorted nonzeros) gives the same values
    Ks = orc.kernel(sp.csr_matrix(A), sp.csr_matrix(B), gamma, kind, degree,
                    coef0)
    np.testing.assert_allclose(Ks, ref, rtol=1e-12, atol=1e-13)
    rows = orc.kernel_rows(B, gamma, [0, 4, 8], 0, kind, degree, coef0)
    ref_r = _sk_kernel(kind, B[[0, 4, 8]], B, gamma, degree, coef0)
    np.testing.assert_allclose(rows, ref_r, rtol=1e-12, atol=1e-13)


def test_kernel_worked_numbers(orc):
    # u = (1, 2), v = (3, -1): u.v = 1, |u|^2 = 5
    u = np.array([[1.0, 2.0]], np.float32)
    v = np.array([[3.0, -1.0]], np.float32)
    assert orc.kernel(u, v, 0.0, LINEAR)[0, 0] == 1.0
    assert orc.kernel(u, u, 0.0, LINEAR)[0, 0] == 5.0
    # (0.5 * 1 + 1)^3 = 3.375 and (0.5 * 5 + 1)^2 = 12.25
    assert orc.kernel(u, v, 0.5, POLY, 3, 1.0)[0, 0] == pytest.approx(3.375,
                                                                     rel=1e-15)
    assert orc.kernel(u, u, 0.5, POLY, 2, 1.0)[0, 0] == pytest.approx(12.25,
                                                                     rel=1e-15)
    # tanh(0.5 + 1) = tanh(1.5)
    assert orc.kernel(u, v, 0.5, SIGMOID, 3, 1.0)[0, 0] == pytest.approx(
        0.9051482536448664, rel=1e-14)


@pytest.mark.parametrize("kind,gamma,degree,coef0,C", [
    (LINEAR, 0.0, 3, 0.0, 100.0), (LINEAR, 0.0, 3, 0.0, 0.1),
    (POLY, 0.5, 3, 1.0, 100.0), (POLY, 0.5, 2, 0.0, 1e-3)])
def test_two_point_closed_form(orc, kind, gamma, degree, coef0, C):
    # x1 (+1), x2 (-1): alpha_1 = alpha_2 = min(C, 2 / a) with
    # a = K11 + K22 - 2 K12; f = a alpha^2 / 2 - 2 alpha; when alpha is free
    # the two margin conditions give b = 1 - alpha (K11 - K12)
    X = np.array([[0.2, 0.1], [1.0, 0.5]], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    K = _sk_kernel(kind, X, X, gamma, degree, coef0)
    a = K[0, 0] + K[1, 1] - 2 * K[0, 1]
    al = min(C, 2.0 / a)
    r = orc.train(X, y, Params(C_SVC, C=C, gamma=gamma, tol=1e-12,
                               kernel=kind, degree=degree, coef0=coef0))
    np.testing.assert_allclose(r.alpha, [al, al], rtol=1e-12)
    assert r.obj == pytest.approx(0.5 * a * al * al - 2 * al, rel=1e-12)
    if al < C:
        assert r.b == pytest.approx(1 - al * (K[0, 0] - K[0, 1]), abs=1e-10)
    # one maximal-violating-pair step from alpha = 0 lands on the optimum
    # exactly: its length is (m - M) / a = 2 / a (pins the pair curvature
    # K11 + K22 - 2 K12 of a kernel whose K(x, x) is not 1)
    p1 = Params(C_SVC, C=C, gamma=gamma, tol=1e-12, kernel=kind,
                degree=degree, coef0=coef0)
    r1 = orc.solve(X, y, p1, np.zeros(2), np.zeros(2), max_steps=1)
    assert r1.iters == 1
    np.testing.assert_allclose(r1.alpha, [al, al], rtol=1e-13)


BF_CASES = [
    # kind, gamma, degree, coef0, type, n, d, C, eps, seed
    (LINEAR, 0.0, 3, 0.0, "svc", 5, 6, 1.0, 0.0, 41),
    (LINEAR, 0.0, 3, 0.0, "svc", 6, 7, 10.0, 0.0, 42),
    (POLY, 0.5, 3, 1.0, "svc", 6, 3, 1.0, 0.0, 43),
    (POLY, 0.3, 2, 1.0, "svc", 7, 3, 5.0, 0.0, 44),
    (LINEAR, 0.0, 3, 0.0, "svr", 3, 4, 2.0, 0.1, 45),
    (POLY, 0.5, 3, 1.0, "svr", 4, 3, 1.0, 0.05, 46),
]


@pytest.mark.parametrize("kind,gamma,degree,coef0,typ,n,d,C,eps,seed",
                         BF_CASES)
def test_exact_optimum_other_kernels(orc, kind, gamma, degree, coef0, typ, n,
                                     d, C, eps, seed):
    X, y = tiny(n, d, seed, typ)
    K = _sk_kernel(kind, X, X, gamma, degree, coef0)
    assert np.linalg.eigvalsh(K).min() > 1e-8  # positive definite: unique
    if typ == "svc":
        type_ = C_SVC
        yy = np.where(y > 0, 1.0, -1.0)
        smp = np.arange(n)
        p = -np.ones(n)
    else:
        type_ = EPS_SVR
        z = y.astype(np.float64)
        yy = np.concatenate([np.ones(n), -np.ones(n)])
        smp = np.concatenate([np.arange(n), np.arange(n)])
        p = np.concatenate([eps - z, eps + z])
    Q = yy[:, None] * yy[None, :] * K[np.ix_(smp, smp)]
    f_star, a_star = brute_force(Q, p, yy, C)
    r = orc.train(X, y, Params(type_, C=C, eps=eps, gamma=gamma, tol=1e-11,
                               kernel=kind, degree=degree, coef0=coef0))
    assert r.status == 0
    f_or = 0.5 * r.alpha @ Q @ r.alpha + p @ r.alpha
    assert r.obj == pytest.approx(f_or, rel=1e-10, abs=1e-12)
    assert f_or == pytest.approx(f_star, rel=1e-9, abs=1e-10)
    c_star = np.bincount(smp, weights=yy * a_star, minlength=n)
    c_or = np.bincount(smp, weights=yy * r.alpha, minlength=n)
    np.testing.assert_allclose(c_or, c_star, atol=1e-6 * max(C, 1))


def _sk_name(kind):
    return {LINEAR: "linear", POLY: "poly", SIGMOID: "sigmoid"}[kind]


@pytest.mark.parametrize("kind,gamma,degree,coef0,C", [
    (LINEAR, 0.0, 3, 0.0, 0.5), (POLY, 0.05, 3, 1.0, 1.0),
    (SIGMOID, 0.01, 3, -0.5, 1.0)])
def test_svc_endpoint_vs_libsvm(orc, kind, gamma, degree, coef0, C):
    w = workloads.c1(n=600, n_test=300)
    p = Params(C_SVC, C=C, gamma=gamma, tol=1e-3, kernel=kind, degree=degree,
               coef0=coef0)
    r = orc.train(w.X, w.y, p)
    assert r.status == 0
    D = orc.model_decision(w.X, w.y, p, r, w.Xt)
    lib = SVC(C=C, kernel=_sk_name(kind), gamma=gamma if gamma > 0 else 1.0,
              degree=degree, coef0=coef0, tol=1e-3, shrinking=False)
    lib.fit(w.X.astype(np.float64), w.y)
    Dl = lib.decision_function(w.Xt.astype(np.float64))
    cl = np.zeros(w.n)
    cl[lib.support_] = lib.dual_coef_[0]
    K = _sk_kernel(kind, w.X, w.X, gamma, degree, coef0)
    f_lib = 0.5 * cl @ K @ cl - np.abs(cl).sum()
    assert r.obj == pytest.approx(f_lib, rel=1e-4)
    np.testing.assert_allclose(D, Dl, atol=3e-3 * max(1.0, np.abs(Dl).max()))
    assert np.mean(np.sign(D) == np.sign(Dl)) >= 0.99


def test_svr_endpoint_vs_libsvm_poly(orc):
    w = workloads.c2(n=800, n_test=300)
    gamma, degree, coef0 = 0.05, 3, 1.0
    p = Params(EPS_SVR, C=w.C, eps=w.eps, gamma=gamma, tol=1e-3, kernel=POLY,
               degree=degree, coef0=coef0)
    r = orc.train(w.X, w.y, p)
    assert r.status == 0
    D = orc.model_decision(w.X, w.y, p, r, w.Xt)
    lib = SVR(C=w.C, epsilon=w.eps, kernel="poly", gamma=gamma, degree=degree,
              coef0=coef0, tol=1e-3, shrinking=False)
    lib.fit(w.X.astype(np.float64), w.y.astype(np.float64))
    Dl = lib.predict(w.Xt.astype(np.float64))
    cl = np.zeros(w.n)
    cl[lib.support_] = lib.dual_coef_[0]
    c = orc.coefficients(EPS_SVR, w.n, w.y, r.alpha)
    K = _sk_kernel(POLY, w.X, w.X, gamma, degree, coef0)
    z = w.y.astype(np.float64)
    f_lib = 0.5 * cl @ K @ cl + w.eps * np.abs(cl).sum() - z @ cl
    f_or = 0.5 * c @ K @ c + w.eps * np.abs(c).sum() - z @ c
    assert r.obj == pytest.approx(f_or, rel=1e-9)
    assert f_or == pytest.approx(f_lib, rel=1e-4)
    np.testing.assert_allclose(D, Dl, atol=3e-3)
