"""The end of a training on the GPU: responses recomputed from alpha, the gap
re-tested on them, bias (free-key mean, else the
midpoint) and objective, and the status when the
gap stays above tol.

Through the svm_test_finish hook, from states the oracle reaches in a given
number of pair steps (not converged, with free and bounded variables, so
that the free-key mean and the midpoint (m + M) / 2 differ).
"""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _state(w, steps):
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    N = oracle.num_vars(w.type, w.n)
    r = oracle.solve(w.X, w.y, p, np.zeros(N), np.zeros(w.n),
                     max_steps=steps)
    assert r.iters == steps
    return p, r.alpha


@pytest.mark.parametrize("name,n,steps", [("C1", 700, 60), ("C2", 500, 80)])
def test_finish_without_passes_reports_recomputed_state(name, n, steps):
    w = workloads.make(name, n=n, n_test=10)
    p, alpha = _state(w, steps)
    Fo = oracle.responses(w.X, w.y, p, alpha)
    ref = oracle.state_summary(w.y, p, alpha, Fo, d=w.d)
    assert ref.gap > w.tol and ref.n_free > 0
    # the free-key mean and the midpoint are far apart in this state
    assert abs(ref.b - 0.5 * (ref.m + ref.M)) > 1e-2
    s = nv.Solver(w.X, w.y, type=w.type, C=w.C, epsilon=w.eps,
                  gamma=w.gamma, tol=w.tol)
    # responses deliberately wrong: the hook must recompute them from alpha
    s.set_state(alpha, np.zeros(w.n))
    gap, b, obj, status = s.finish(max_passes=0)
    assert status == nv.SVM_W_NOT_CONVERGED
    scale = max(1.0, float(np.max(np.abs(Fo))))
    assert gap == pytest.approx(ref.gap, abs=1e-5 * scale)
    assert b == pytest.approx(ref.b, abs=1e-5 * scale)
    assert obj == pytest.approx(ref.obj, rel=1e-6)


@pytest.mark.parametrize("name,n,steps", [("C1", 700, 60), ("C2", 500, 80)])
def test_finish_with_passes_runs_to_tol(name, n, steps):
    w = workloads.make(name, n=n, n_test=10)
    p, alpha = _state(w, steps)
    s = nv.Solver(w.X, w.y, type=w.type, C=w.C, epsilon=w.eps,
                  gamma=w.gamma, tol=w.tol)
    s.set_state(alpha, np.zeros(w.n))
    gap, b, obj, status = s.finish(max_passes=3)
    assert status == nv.SVM_OK
    assert gap <= w.tol
    a2, F2 = s.get_state()
    Fo = oracle.responses(w.X, w.y, p, a2)
    ref = oracle.state_summary(w.y, p, a2, Fo, d=w.d)
    assert ref.gap <= w.tol * 1.01
    assert b == pytest.approx(ref.b, abs=1e-4)
    full = oracle.train(w.X, w.y, p)
    assert obj == pytest.approx(full.obj, rel=1e-4)


def test_converged_state_is_accepted_at_once():
    # the oracle's optimum at a tol well inside the solver's
    w = workloads.c1(n=600, n_test=10)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=1e-5)
    r = oracle.train(w.X, w.y, p)
    s = nv.Solver(w.X, w.y, type=C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    s.set_state(r.alpha, np.zeros(w.n))
    gap, b, obj, status = s.finish(max_passes=0)
    assert status == nv.SVM_OK and gap <= w.tol
    assert b == pytest.approx(r.b, abs=1e-4)
    assert obj == pytest.approx(r.obj, rel=1e-6)
    a2, _ = s.get_state()
    assert np.array_equal(a2, r.alpha)  # nothing re-run
