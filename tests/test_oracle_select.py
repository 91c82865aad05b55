"""Pins for the oracle's working-set selection and subproblem (Section 3).

The selection is checked against a direct sort of keys computed here from
scikit-learn's kernel; the subproblem against (a) one maximal-violating-pair
step of the full solver when the working set is the pair, and (b) the exact
optimum of the problem restricted to the working set, by enumeration.
"""
import itertools

import numpy as np
import pytest
from sklearn.metrics.pairwise import rbf_kernel

from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import workloads


def _vars(w):
    n = w.n
    if w.type == C_SVC:
        yy = np.where(w.y > 0, 1.0, -1.0)
        r = yy.copy()
        smp = np.arange(n)
    else:
        z = w.y.astype(np.float64)
        yy = np.concatenate([np.ones(n), -np.ones(n)])
        r = np.concatenate([z - w.eps, z + w.eps])
        smp = np.concatenate([np.arange(n), np.arange(n)])
    return yy, r, smp


def _state(orc, w, steps):
    """The state after `steps` pair steps from alpha = 0; steps = 0 is the
    start state itself (alpha = 0, F = 0), built here: solve's max_steps = 0
    means "no cap"."""
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    N = orc.num_vars(w.type, w.n)
    if steps == 0:
        return p, np.zeros(N), np.zeros(w.n)
    res = orc.solve(w.X, w.y, p, np.zeros(N), np.zeros(w.n), max_steps=steps)
    assert res.iters == steps
    return p, res.alpha, res.F


def _expected_ws(w, alpha, F, q):
    yy, r, smp = _vars(w)
    v = r - F[smp]
    up = ((yy > 0) & (alpha < w.C)) | ((yy < 0) & (alpha > 0))
    lo = ((yy > 0) & (alpha > 0)) | ((yy < 0) & (alpha < w.C))
    t = np.arange(len(v))
    U = sorted(t[up], key=lambda i: (-v[i], i))[: q // 2]
    L = sorted(t[lo], key=lambda i: (v[i], i))[: q // 2]
    B = []
    for k in range(q // 2):
        for side in (U, L):
            if k < len(side) and side[k] not in B:
                B.append(side[k])
    m = v[U[0]] if U else -np.inf
    M = v[L[0]] if L else np.inf
    return np.array(B), m, M


@pytest.mark.parametrize("name,steps,q", [("C1", 0, 16), ("C1", 40, 16),
                                          ("C1", 40, 2), ("C2", 60, 16),
                                          ("C2", 7, 6)])
def test_select_matches_sorted_keys(orc, name, steps, q):
    w = workloads.make(name, n=400, n_test=10)
    p, alpha, F = _state(orc, w, steps)
    B, m, M = orc.select(w.y, p, alpha, F, q, d=w.d)
    Be, me, Me = _expected_ws(w, alpha, F, q)
    assert list(B) == list(Be)
    assert m == me and M == Me


def test_pair_subproblem_equals_one_smo_step(orc):
    w = workloads.c1(n=300, n_test=10)
    p, alpha, F = _state(orc, w, 25)
    B, m, M = orc.select(w.y, p, alpha, F, 2, d=w.d)
    aB, steps = orc.subproblem(w.X, w.y, p, alpha, F, B, 0.0, 1)
    assert steps == 1
    nxt = orc.solve(w.X, w.y, p, alpha, F, max_steps=1)
    exp = alpha.copy()
    exp[B] = aB
    assert np.array_equal(nxt.alpha, exp)


def _restricted_optimum(Q, G, yy, alpha, B, C):
    """min_d 1/2 d^T Q_BB d + G_B^T d, y_B^T d = 0, 0 <= alpha_B + d <= C."""
    QB = Q[np.ix_(B, B)]
    gB = G[B]
    yB = yy[B]
    a0 = alpha[B]
    best = None
    for assign in itertools.product((0, 1, 2), repeat=len(B)):
        a = np.array([0.0 if s == 0 else C for s in assign])
        f = [k for k, s in enumerate(assign) if s == 2]
        fx = [k for k, s in enumerate(assign) if s != 2]
        if f:
            m = len(f)
            A = np.zeros((m + 1, m + 1))
            A[:m, :m] = QB[np.ix_(f, f)]
            A[:m, m] = yB[f]
            A[m, :m] = yB[f]
            # stationarity of the restricted problem in terms of the new a_B
            rhs = np.zeros(m + 1)
            lin = gB - QB @ a0
            rhs[:m] = -lin[f] - (QB[np.ix_(f, fx)] @ a[fx] if fx else 0.0)
            rhs[m] = yB @ a0 - (yB[fx] @ a[fx] if fx else 0.0)
            try:
                sol = np.linalg.solve(A, rhs)
            except np.linalg.LinAlgError:
                continue
            if not np.allclose(A @ sol, rhs, atol=1e-9):
                continue
            a[f] = sol[:m]
            if np.any(a < -1e-12) or np.any(a > C + 1e-12):
                continue
        if abs(yB @ (a - a0)) > 1e-9:
            continue
        dd = a - a0
        obj = 0.5 * dd @ QB @ dd + gB @ dd
        if best is None or obj < best[0]:
            best = (obj, a)
    return best


@pytest.mark.parametrize("name,steps,q", [("C1", 30, 6), ("C2", 30, 6),
                                          ("C1", 0, 4)])
def test_subproblem_reaches_restricted_optimum(orc, name, steps, q):
    w = workloads.make(name, n=200, n_test=10)
    p, alpha, F = _state(orc, w, steps)
    B, _, _ = orc.select(w.y, p, alpha, F, q, d=w.d)
    yy, r, smp = _vars(w)
    K = rbf_kernel(w.X.astype(np.float64), gamma=w.gamma)
    Q = yy[:, None] * yy[None, :] * K[np.ix_(smp, smp)]
    G = -yy * (r - F[smp])
    f_star, a_star = _restricted_optimum(Q, G, yy, alpha, B, w.C)
    aB, steps_taken = orc.subproblem(w.X, w.y, p, alpha, F, B, 1e-12, 10000)
    dd = aB - alpha[B]
    QB = Q[np.ix_(B, B)]
    f_or = 0.5 * dd @ QB @ dd + G[B] @ dd
    assert f_or == pytest.approx(f_star, rel=1e-8, abs=1e-10)
    assert abs(yy[B] @ dd) < 1e-10
    assert np.all(aB >= 0) and np.all(aB <= w.C)


# ---------------------------------------------------------------------------
# Tie-break (lowest variable index among equal keys) pinned by states whose
# working set follows from the labels alone.
# ---------------------------------------------------------------------------

def _interleave(U, L):
    B = []
    for k in range(max(len(U), len(L))):
        for side in (U, L):
            if k < len(side) and side[k] not in B:
                B.append(side[k])
    return B


@pytest.mark.parametrize("q", [2, 6, 16])
def test_select_alpha0_svc_takes_lowest_indices(orc, q):
    # At alpha = 0 and F = 0 every C-SVC key is v_t = y_t: I_up is the +1
    # class with key +1, I_low the -1 class with key -1.  Every key of a
    # side ties, so the q/2 largest (smallest) are the q/2 lowest indices
    # of each class, and m = 1, M = -1.
    w = workloads.c1(n=400, n_test=10)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    B, m, M = orc.select(w.y, p, np.zeros(w.n), np.zeros(w.n), q, d=w.d)
    pos = [int(i) for i in np.nonzero(w.y > 0)[0][: q // 2]]
    neg = [int(i) for i in np.nonzero(w.y < 0)[0][: q // 2]]
    assert list(B) == _interleave(pos, neg)
    assert (m, M) == (1.0, -1.0)


@pytest.mark.parametrize("q", [2, 6, 16])
def test_select_alpha0_svr_ties_on_targets(orc, q):
    # eps-SVR at alpha = 0, F = 0: copy (i,+) is in I_up with key z_i - eps,
    # copy (i,-) (variable n + i) in I_low with key z_i + eps.  Targets in
    # {0, 1}: the largest up keys are the copies (i,+) with z_i = 1, the
    # smallest low keys the copies (i,-) with z_i = 0, each in increasing
    # index order.
    rng = np.random.default_rng(5)
    n = 300
    z = (rng.random(n) < 0.4).astype(np.float32)
    eps = 0.1
    p = Params(EPS_SVR, C=1.0, eps=eps, gamma=0.5, tol=1e-3)
    B, m, M = orc.select(z, p, np.zeros(2 * n), np.zeros(n), q, d=4)
    up = [int(i) for i in np.nonzero(z == 1)[0][: q // 2]]
    lo = [int(n + i) for i in np.nonzero(z == 0)[0][: q // 2]]
    assert list(B) == _interleave(up, lo)
    assert m == np.float64(1.0) - eps and M == 0.0 + eps


@pytest.mark.parametrize("q", [4, 16])
def test_select_tied_keys_by_counting(orc, q):
    # A state with bounded and free variables and keys on a coarse grid
    # (many ties): the working set by brute force, each entry's place in a
    # side being the number of entries that precede it (larger key for
    # I_up, smaller for I_low, equal keys ordered by index).
    w = workloads.c1(n=240, n_test=10)
    rng = np.random.default_rng(11)
    C = w.C
    alpha = rng.choice([0.0, 0.5 * C, C], size=w.n)
    F = np.round(rng.normal(size=w.n) * 2) / 4  # keys on a 0.25 grid
    p = Params(C_SVC, C=C, gamma=w.gamma, tol=w.tol)
    B, m, M = orc.select(w.y, p, alpha, F, q, d=w.d)
    yy = np.where(w.y > 0, 1.0, -1.0)
    v = yy - F
    up = [t for t in range(w.n)
          if (yy[t] > 0 and alpha[t] < C) or (yy[t] < 0 and alpha[t] > 0)]
    lo = [t for t in range(w.n)
          if (yy[t] > 0 and alpha[t] > 0) or (yy[t] < 0 and alpha[t] < C)]

    def place(side, t, sign):
        return sum(1 for u in side
                   if sign * v[u] > sign * v[t] or (v[u] == v[t] and u < t))

    U = [None] * (q // 2)
    for t in up:
        k = place(up, t, 1.0)
        if k < q // 2:
            U[k] = t
    L = [None] * (q // 2)
    for t in lo:
        k = place(lo, t, -1.0)
        if k < q // 2:
            L[k] = t
    assert list(B) == _interleave(U, L)
    assert m == max(v[up]) and M == min(v[lo])
    # the grid really ties entries inside the selected prefix
    assert len(set(v[U])) < len(U) or len(set(v[L])) < len(L)
