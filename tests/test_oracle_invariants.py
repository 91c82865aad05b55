"""Oracle pinned by the invariants of Eq. 2 on the small workloads.

Feasibility (box and equality constraint), the KKT gap at exit, responses
recomputed from scratch (which catches a wrong incremental update), the
objective recomputed from scikit-learn's kernel, a monotone objective per
SMO step, one active copy per sample for eps-SVR, and free variables sitting
on the margin / tube edge.
"""
import numpy as np
import pytest
from sklearn.metrics.pairwise import rbf_kernel

from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import workloads


def _params(w, tol=None):
    return Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma,
                  tol=w.tol if tol is None else tol)


def _check_state(orc, w, r, tol):
    p = _params(w)
    n = w.n
    N = orc.num_vars(w.type, n)
    a = r.alpha
    assert a.shape == (N,)
    assert np.all(a >= 0) and np.all(a <= w.C)
    yy = (np.where(w.y > 0, 1.0, -1.0) if w.type == C_SVC
          else np.concatenate([np.ones(n), -np.ones(n)]))
    assert abs(yy @ a) <= 1e-10 * w.C * N
    assert r.status == 0 and r.gap <= tol
    F = orc.responses(w.X, w.y, p, a)
    np.testing.assert_allclose(r.F, F, rtol=1e-9, atol=1e-9)
    # objective with an independent kernel
    K = rbf_kernel(w.X.astype(np.float64), gamma=w.gamma)
    c = orc.coefficients(w.type, n, w.y, a)
    if w.type == C_SVC:
        lin = -a.sum()
    else:
        z = w.y.astype(np.float64)
        lin = (w.eps - z) @ a[:n] + (w.eps + z) @ a[n:]
    f = 0.5 * c @ K @ c + lin
    assert r.obj == pytest.approx(f, rel=1e-9)
    # free variables lie within tol of the bias (margin / tube edge)
    D = K @ c + r.b
    if w.type == C_SVC:
        free = (a > 0) & (a < w.C)
        np.testing.assert_allclose(D[free], yy[free], atol=tol + 1e-9)
    else:
        z = w.y.astype(np.float64)
        fp = (a[:n] > 0) & (a[:n] < w.C)
        fm = (a[n:] > 0) & (a[n:] < w.C)
        np.testing.assert_allclose(D[fp], z[fp] - w.eps, atol=tol + 1e-9)
        np.testing.assert_allclose(D[fm], z[fm] + w.eps, atol=tol + 1e-9)
    return c


def test_c1_invariants(orc):
    w = workloads.c1()
    r = orc.train(w.X, w.y, _params(w))
    _check_state(orc, w, r, w.tol)
    assert 100 < r.n_sv < 1000
    # accuracy on the held-out set near the Bayes rate (1.3% error)
    D = orc.model_decision(w.X, w.y, _params(w), r, w.Xt)
    acc = np.mean(np.where(D >= 0, 1.0, -1.0) == w.yt)
    assert acc > 0.97


def test_c2_subsample_invariants(orc):
    w = workloads.c2(n=1500, n_test=500)
    r = orc.train(w.X, w.y, _params(w))
    c = _check_state(orc, w, r, w.tol)
    n = w.n
    # eps > 0: a sample never keeps both copies active at the optimum
    both = np.minimum(r.alpha[:n], r.alpha[n:])
    assert np.max(both) <= 1e-9
    assert np.count_nonzero(c) == r.n_sv
    D = orc.model_decision(w.X, w.y, _params(w), r, w.Xt)
    mse = np.mean((D - w.yt) ** 2)
    assert mse < 0.6 * np.var(w.yt)  # explains a good part of the variance


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_objective_monotone_per_step(orc, name):
    w = workloads.make(name, n=300, n_test=10)
    p = _params(w)
    N = orc.num_vars(w.type, w.n)
    a = np.zeros(N)
    F = np.zeros(w.n)
    prev = 0.0
    for _ in range(150):
        r = orc.solve(w.X, w.y, p, a, F, max_steps=1)
        assert r.obj <= prev + 1e-12
        prev = r.obj
        a, F = r.alpha, r.F
        if r.iters == 0:
            break


def test_max_iter_status(orc):
    w = workloads.c1(n=400, n_test=10)
    p = _params(w)
    p.max_iter = 5
    r = orc.train(w.X, w.y, p)
    assert r.status == 1 and r.iters == 5 and r.gap > w.tol


def test_threads_do_not_change_bits(orc):
    w = workloads.c1(n=500, n_test=100)
    p1 = _params(w)
    p1.threads = 1
    p4 = _params(w)
    p4.threads = 4
    r1 = orc.train(w.X, w.y, p1)
    r4 = orc.train(w.X, w.y, p4)
    assert np.array_equal(r1.alpha, r4.alpha)
    assert np.array_equal(r1.F, r4.F)
