"""Oracle pinned by the exact optimum of Eq. 2 on tiny problems.

The exact optimum comes from active-set enumeration, independent of SMO:
each variable is put at 0, at C or free; for the free ones the stationarity
conditions (Qa + p)_t + y_t b = 0 together with y^T a = 0 form a linear
system; feasible solutions are kept and the one with the smallest objective
is the global minimum (the problem is convex).  Q is built with
scikit-learn's rbf_kernel, not with the oracle's kernel.
"""
import itertools

import numpy as np
import pytest
from sklearn.metrics.pairwise import rbf_kernel

from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd.workloads import tiny


def _problem(X, y, type_, C, eps, gamma):
    K = rbf_kernel(X.astype(np.float64), gamma=gamma)
    n = len(X)
    if type_ == C_SVC:
        yy = np.where(y > 0, 1.0, -1.0)
        Q = yy[:, None] * yy[None, :] * K
        p = -np.ones(n)
        smp = np.arange(n)
    else:
        z = y.astype(np.float64)
        yy = np.concatenate([np.ones(n), -np.ones(n)])
        smp = np.concatenate([np.arange(n), np.arange(n)])
        Q = yy[:, None] * yy[None, :] * K[np.ix_(smp, smp)]
        p = np.concatenate([eps - z, eps + z])
    return Q, p, yy, smp


def brute_force(Q, p, yy, C):
    N = len(p)
    best = None
    for assign in itertools.product((0, 1, 2), repeat=N):  # 0: lo, 1: C, 2: free
        a = np.array([0.0 if s == 0 else C for s in assign])
        free = [t for t, s in enumerate(assign) if s == 2]
        if free:
            f = np.array(free)
            fixed = np.array([t for t in range(N) if assign[t] != 2], int)
            m = len(f)
            A = np.zeros((m + 1, m + 1))
            A[:m, :m] = Q[np.ix_(f, f)]
            A[:m, m] = yy[f]
            A[m, :m] = yy[f]
            rhs = np.zeros(m + 1)
            rhs[:m] = -p[f] - (Q[np.ix_(f, fixed)] @ a[fixed] if len(fixed) else 0)
            rhs[m] = -(yy[fixed] @ a[fixed]) if len(fixed) else 0.0
            try:
                sol = np.linalg.solve(A, rhs)
            except np.linalg.LinAlgError:
                continue
            if not np.allclose(A @ sol, rhs, atol=1e-9):
                continue
            a[f] = sol[:m]
            if np.any(a[f] < -1e-12) or np.any(a[f] > C + 1e-12):
                continue
        if abs(yy @ a) > 1e-9:
            continue
        obj = 0.5 * a @ Q @ a + p @ a
        if best is None or obj < best[0] - 1e-15:
            best = (obj, a.copy())
    return best


CASES = [
    ("svc", 5, 3, 1.0, 0.0, 0.4, 11),
    ("svc", 6, 2, 0.5, 0.0, 1.0, 12),
    ("svc", 7, 4, 10.0, 0.0, 0.25, 13),
    ("svc", 6, 3, 3.0, 0.0, 0.7, 14),
    ("svr", 3, 2, 2.0, 0.1, 0.5, 21),
    ("svr", 4, 3, 1.0, 0.05, 0.8, 22),
    ("svr", 4, 2, 10.0, 0.2, 0.3, 23),
]


@pytest.mark.parametrize("kind,n,d,C,eps,gamma,seed", CASES)
def test_oracle_reaches_exact_optimum(orc, kind, n, d, C, eps, gamma, seed):
    X, y = tiny(n, d, seed, kind)
    type_ = C_SVC if kind == "svc" else EPS_SVR
    Q, p, yy, smp = _problem(X, y, type_, C, eps, gamma)
    f_star, a_star = brute_force(Q, p, yy, C)

    r = orc.train(X, y, Params(type_, C=C, eps=eps, gamma=gamma, tol=1e-11))
    assert r.status == 0
    # objective computed independently from the oracle's own bookkeeping
    f_or = 0.5 * r.alpha @ Q @ r.alpha + p @ r.alpha
    assert r.obj == pytest.approx(f_or, rel=1e-10, abs=1e-12)
    assert f_or == pytest.approx(f_star, rel=1e-9, abs=1e-10)
    assert f_or >= f_star - 1e-10
    # the RBF Gram matrix of distinct points is positive definite, so the
    # expansion coefficients of the optimum are unique
    c_star = np.bincount(smp, weights=yy * a_star, minlength=n)
    c_or = np.bincount(smp, weights=yy * r.alpha, minlength=n)
    np.testing.assert_allclose(c_or, c_star, atol=1e-6 * max(C, 1))

    # at the loose tolerance the objective is still close to the optimum
    r3 = orc.train(X, y, Params(type_, C=C, eps=eps, gamma=gamma, tol=1e-3))
    f3 = 0.5 * r3.alpha @ Q @ r3.alpha + p @ r3.alpha
    assert f_star - 1e-12 <= f3 <= f_star + 1e-3 * len(p) * C


@pytest.mark.parametrize("kind,n,d,C,eps,gamma,seed", CASES[:4])
def test_bias_matches_free_multiplier(orc, kind, n, d, C, eps, gamma, seed):
    # for a free variable at the optimum (Qa + p)_t = -y_t b
    X, y = tiny(n, d, seed, kind)
    Q, p, yy, smp = _problem(X, y, C_SVC, C, eps, gamma)
    _, a_star = brute_force(Q, p, yy, C)
    free = np.nonzero((a_star > 1e-9) & (a_star < C - 1e-9))[0]
    r = orc.train(X, y, Params(C_SVC, C=C, gamma=gamma, tol=1e-11))
    if len(free):
        G = Q @ a_star + p
        b_star = np.mean(-yy[free] * G[free])
        assert r.b == pytest.approx(b_star, abs=1e-7)


def test_duplicate_points_degenerate_pair(orc):
    # x_2 == x_0: the pair curvature K00 + K22 - 2K02 is 0 (it is
    # floored at tau = 1e-12)
    X, y = tiny(6, 3, 31, "svc", duplicates=True)
    y[2] = -y[0]
    Q, p, yy, _ = _problem(X, y, C_SVC, 1.0, 0.0, 0.5)
    f_star, _ = brute_force(Q, p, yy, 1.0)
    r = orc.train(X, y, Params(C_SVC, C=1.0, gamma=0.5, tol=1e-10))
    assert r.status == 0
    f_or = 0.5 * r.alpha @ Q @ r.alpha + p @ r.alpha
    assert f_or == pytest.approx(f_star, rel=1e-8, abs=1e-10)
    assert np.all(r.alpha >= 0) and np.all(r.alpha <= 1.0)
