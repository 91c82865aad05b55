"""Oracle pinned by closed-form optima of Eq. 2 on 2- and 3-point problems.

Each closed form is derived by hand from the dual of Eq. 2 (Section 3):
symmetry reduces the problem to one scalar, whose minimiser is a clipped
quotient.  A dropped term, a wrong sign of p or a swapped SVR copy changes
these numbers.
"""
import math

import numpy as np
import pytest

from oracle import C_SVC, EPS_SVR, Params

TIGHT = 1e-10


def _k(a, b, gamma):
    return math.exp(-gamma * sum((float(x) - float(z)) ** 2
                                 for x, z in zip(a, b)))


@pytest.mark.parametrize("C", [1.0, 10.0, 0.3])
def test_two_point_svc(orc, C):
    # x1 = (0,0) class +1, x2 = (1,0.5) class -1.  With a1 = a2 = a the dual
    # objective is a^2 (1-k) - 2a, minimised at a = 1/(1-k), clipped to C.
    X = np.array([[0.0, 0.0], [1.0, 0.5]], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    g = 0.5
    k = _k(X[0], X[1], g)
    assert k == pytest.approx(0.535261, abs=1e-6)
    a = min(C, 1.0 / (1.0 - k))
    r = orc.train(X, y, Params(C_SVC, C=C, gamma=g, tol=TIGHT))
    assert r.status == 0
    np.testing.assert_allclose(r.alpha, [a, a], rtol=1e-9)
    assert r.obj == pytest.approx(a * a * (1 - k) - 2 * a, rel=1e-9)
    assert r.b == pytest.approx(0.0, abs=1e-9)
    D = orc.model_decision(X, y, Params(C_SVC, C=C, gamma=g), r, X)
    if a < C:  # both are free margin vectors: D = y exactly
        np.testing.assert_allclose(D, y, atol=1e-8)


def test_two_point_svc_worked_numbers(orc):
    X = np.array([[0.0, 0.0], [1.0, 0.5]], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    r1 = orc.train(X, y, Params(C_SVC, C=1.0, gamma=0.5, tol=TIGHT))
    assert r1.obj == pytest.approx(-1.535261, abs=1e-6)
    r10 = orc.train(X, y, Params(C_SVC, C=10.0, gamma=0.5, tol=TIGHT))
    assert r10.alpha[0] == pytest.approx(2.151747, abs=1e-6)
    assert r10.obj == pytest.approx(-2.151747, abs=1e-6)


@pytest.mark.parametrize("C", [100.0, 1.0, 3.0])
def test_three_point_symmetric_svc(orc, C):
    # x3 = 0 (class -1) between x1 = u and x2 = -u (class +1).  Symmetry
    # gives a = (a, a, 2a) and objective a^2 (3 + k' - 4k) - 4a.
    u = np.array([0.8, 0.3])
    X = np.array([u, -u, [0.0, 0.0]], np.float32)
    y = np.array([1.0, 1.0, -1.0], np.float32)
    g = 0.5
    k = _k(X[0], X[2], g)
    kp = _k(X[0], X[1], g)
    a = min(2.0 / (3.0 + kp - 4.0 * k), C / 2.0)
    r = orc.train(X, y, Params(C_SVC, C=C, gamma=g, tol=TIGHT))
    np.testing.assert_allclose(r.alpha, [a, a, 2 * a], rtol=1e-8)
    assert r.obj == pytest.approx(a * a * (3 + kp - 4 * k) - 4 * a, rel=1e-9)
    if a < C / 2:
        b = -1.0 + 2.0 * a * (1.0 - k)       # all three free
    else:
        b = 1.0 - a * (1.0 + kp - 2.0 * k)   # x1, x2 free, x3 at C
    assert r.b == pytest.approx(b, abs=1e-8)
    if C == 100.0:
        assert a == pytest.approx(4.391265, abs=1e-6)
        assert b == pytest.approx(1.685727, abs=1e-6)
    if C == 1.0:
        assert b == pytest.approx(1.078079, abs=1e-6)


@pytest.mark.parametrize("z,C", [((2.0, 0.0), 100.0), ((2.0, 0.0), 0.5),
                                 ((0.15, 0.0), 100.0), ((0.0, 1.3), 5.0)])
def test_two_point_svr(orc, z, C):
    # c1 = -c2 = clip((z1 - z2 - 2 eps) / (2 (1-k)), 0, C), b = (z1 + z2)/2
    # (for z1 >= z2; mirrored otherwise).  This pins the sign of the SVR
    # linear term and which copy carries y = +1 (Eq. 1 substituted
    # into Eq. 2).
    X = np.array([[0.0, 0.0], [1.0, 0.5]], np.float32)
    zz = np.array(z, np.float32)
    g, eps = 0.5, 0.1
    k = _k(X[0], X[1], g)
    z1, z2 = float(zz[0]), float(zz[1])
    c = np.clip((abs(z1 - z2) - 2 * eps) / (2 * (1 - k)), 0.0, C)
    sign = 1.0 if z1 >= z2 else -1.0
    p = Params(EPS_SVR, C=C, eps=eps, gamma=g, tol=TIGHT)
    r = orc.train(X, zz, p)
    coef = orc.coefficients(EPS_SVR, 2, zz, r.alpha)
    np.testing.assert_allclose(coef, [sign * c, -sign * c], atol=1e-9)
    assert r.b == pytest.approx((z1 + z2) / 2, abs=1e-9)
    # at most one copy of each sample is active
    assert np.all(np.minimum(r.alpha[:2], r.alpha[2:]) <= 1e-12)
    if z == (2.0, 0.0) and C == 100.0:
        assert c == pytest.approx(1.936573, abs=1e-6)
    if c > 0 and c < C:  # free: the fit sits on the tube edge z -/+ eps
        D = orc.model_decision(X, zz, p, r, X)
        np.testing.assert_allclose(D, [z1 - sign * eps, z2 + sign * eps],
                                   atol=1e-8)


def test_kernel_matches_library_and_identity(orc):
    from sklearn.metrics.pairwise import rbf_kernel
    rng = np.random.default_rng(5)
    A = rng.standard_normal((7, 13)).astype(np.float32)
    B = rng.standard_normal((5, 13)).astype(np.float32)
    K = orc.kernel(A, B, 0.07)
    ref = rbf_kernel(A.astype(np.float64), B.astype(np.float64), gamma=0.07)
    np.testing.assert_allclose(K, ref, rtol=1e-12)
    Kaa = orc.kernel(A, A, 0.07)
    assert np.all(np.diag(Kaa) == 1.0)
    np.testing.assert_allclose(Kaa, Kaa.T, rtol=0, atol=0)
    # factorisation over coordinates: K(a,b) = prod_k exp(-g (a_k-b_k)^2)
    prod = np.ones((7, 5))
    for kk in range(13):
        prod *= orc.kernel(A[:, kk:kk + 1], B[:, kk:kk + 1], 0.07)
    np.testing.assert_allclose(K, prod, rtol=1e-12)


def test_kernel_csr_equals_dense(orc):
    import scipy.sparse as sp
    rng = np.random.default_rng(6)
    A = rng.standard_normal((9, 30)) * (rng.random((9, 30)) < 0.2)
    A = A.astype(np.float32)
    Kd = orc.kernel(A, A, 0.1)
    Ks = orc.kernel(sp.csr_matrix(A), sp.csr_matrix(A), 0.1)
    Km = orc.kernel(sp.csr_matrix(A), A, 0.1)
    np.testing.assert_allclose(Ks, Kd, rtol=1e-14)
    np.testing.assert_allclose(Km, Kd, rtol=1e-14)
    rows = orc.kernel_rows(sp.csr_matrix(A), 0.1, [3, 0])
    np.testing.assert_allclose(rows, Kd[[3, 0]], rtol=1e-14)
