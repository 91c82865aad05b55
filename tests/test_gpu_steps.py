"""Single steps of the HIP path against the CPU oracle from identical states.

Through the C ABI test hooks: kernel rows (1e-5 relative), the working set
and the gap (exact: keys are computed from the same fp64 responses), the
subproblem (same K block, fp64 arithmetic in both), and the response update
(1e-5 relative to max(|F|, 1)).  Shapes cover several 16-row tiles, ragged
row and feature tails, and both problem types.
"""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu

SHAPES = [  # name, n, d override (None: the workload's d)
    ("C1", 333, None),
    ("C1", 1000, 7),
    ("C2", 517, None),
    ("C3", 900, None),
    ("C3", 130, 33),
]


def _work(name, n, d):
    w = workloads.make(name, n=n, n_test=50)
    if d is not None:
        w.X = np.ascontiguousarray(w.X[:, :d])
        w.Xt = np.ascontiguousarray(w.Xt[:, :d])
        w.gamma = 1.0 / d
    return w


def _oracle_state(w, steps):
    """The oracle's state after `steps` pair steps from alpha = 0; steps = 0
    is the start state (alpha = 0, F = 0) itself, where every C-SVC key
    ties at +1 or -1 (the oracle's max_steps = 0 would mean no cap)."""
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    N = oracle.num_vars(w.type, w.n)
    if steps == 0:
        return p, np.zeros(N), np.zeros(w.n)
    r = oracle.solve(w.X, w.y, p, np.zeros(N), np.zeros(w.n),
                     max_steps=steps)
    assert r.iters == steps
    return p, r.alpha, r.F


def _solver(w, q=16):
    return nv.Solver(w.X, w.y, type=w.type, C=w.C, epsilon=w.eps,
                     gamma=w.gamma, tol=w.tol, working_set=q)


@pytest.mark.parametrize("name,n,d", SHAPES)
def test_kernel_rows(name, n, d):
    w = _work(name, n, d)
    s = _solver(w)
    rng = np.random.default_rng(n)
    idx = np.concatenate([[0, n - 1], rng.choice(n, 14, replace=False)])
    K = s.rows(idx)
    ref = oracle.kernel_rows(w.X, w.gamma, idx)
    err = np.abs(K - ref) - (1e-5 * np.abs(ref) + 1e-12)
    assert np.max(err) <= 0, np.max(np.abs(K - ref) / (np.abs(ref) + 1e-30))
    # exact self value
    for j, i in enumerate(idx):
        assert K[j, i] == 1.0


@pytest.mark.parametrize("name,n,d", SHAPES)
@pytest.mark.parametrize("steps", [0, 37])
@pytest.mark.parametrize("q", [16, 2, 6])
def test_select_matches_oracle(name, n, d, steps, q):
    w = _work(name, n, d)
    p, alpha, F = _oracle_state(w, steps)
    s = _solver(w, q)
    s.set_state(alpha, F)
    B, m, M = s.select()
    Be, me, Me = oracle.select(w.y, p, alpha, F, q, d=w.d)
    assert m == me and M == Me
    assert list(B) == list(Be)


def _interleave(U, L):
    B = []
    for k in range(max(len(U), len(L))):
        for side in (U, L):
            if k < len(side) and side[k] not in B:
                B.append(side[k])
    return B


@pytest.mark.parametrize("n", [333, 5000])
@pytest.mark.parametrize("q", [2, 6, 16, 32])
def test_select_alpha0_takes_lowest_indices(n, q):
    # alpha = 0, F = 0: every up key is +1 (the +1 class), every low key -1
    # (the -1 class), so the working set is the q/2 lowest indices of each
    # class, interleaved.  Thousands of tied candidates spread over all the
    # row kernel's blocks: the merge must keep the lowest indices.
    w = workloads.c1(n=n, n_test=10)
    s = _solver(w, q)
    s.set_state(np.zeros(n), np.zeros(n))
    B, m, M = s.select()
    pos = [int(i) for i in np.nonzero(w.y > 0)[0][: q // 2]]
    neg = [int(i) for i in np.nonzero(w.y < 0)[0][: q // 2]]
    assert list(B) == _interleave(pos, neg)
    assert (m, M) == (1.0, -1.0)


@pytest.mark.parametrize("q", [2, 16])
def test_select_alpha0_svr_ties(q):
    # eps-SVR at alpha = 0 with targets in {0, 1}: the up side is the copies
    # (i,+) with z_i = 1, the low side the copies (i,-) = n + i with z_i =
    # 0, each in increasing index order.
    rng = np.random.default_rng(5)
    n, d = 3000, 9
    X = rng.normal(size=(n, d)).astype(np.float32)
    z = (rng.random(n) < 0.4).astype(np.float32)
    s = nv.Solver(X, z, type=EPS_SVR, C=1.0, epsilon=0.1, gamma=0.5,
                  tol=1e-3, working_set=q)
    s.set_state(np.zeros(2 * n), np.zeros(n))
    B, m, M = s.select()
    up = [int(i) for i in np.nonzero(z == 1)[0][: q // 2]]
    lo = [int(n + i) for i in np.nonzero(z == 0)[0][: q // 2]]
    assert list(B) == _interleave(up, lo)
    assert m == np.float64(np.float32(1.0)) - 0.1 and M == 0.0 + 0.1


@pytest.mark.parametrize("name,n,d", SHAPES[:4])
def test_subproblem_matches_oracle(name, n, d):
    w = _work(name, n, d)
    p, alpha, F = _oracle_state(w, 25)
    s = _solver(w)
    s.set_state(alpha, F)
    B, m, M = s.select()
    assert len(B) >= 2
    smp = oracle.sample_of(w.type, w.n, B)
    # the GPU's own fp32 kernel block, widened: both sides then do the same
    # fp64 arithmetic on the same numbers
    uniq, inv = np.unique(smp, return_inverse=True)
    Kr = s.rows(uniq).astype(np.float64)
    KBB = Kr[inv][:, smp]
    itol = max(0.1 * (m - M), 0.5 * w.tol)
    aB, steps = s.subproblem(B, itol, 128)
    aBo, steps_o = oracle.subproblem(w.X, w.y, p, alpha, F, B, itol, 128,
                                     KBB=KBB)
    assert steps == steps_o
    np.testing.assert_allclose(aB, aBo, rtol=1e-10, atol=1e-12 * w.C)


@pytest.mark.parametrize("name,n,d", SHAPES)
def test_apply_updates_responses(name, n, d):
    w = _work(name, n, d)
    p, alpha, F = _oracle_state(w, 25)
    B, m, M = oracle.select(w.y, p, alpha, F, 16, d=w.d)
    itol = max(0.1 * (m - M), 0.5 * w.tol)
    aB, _ = oracle.subproblem(w.X, w.y, p, alpha, F, B, itol, 128)
    s = _solver(w)
    s.set_state(alpha, F)
    s.apply(B, aB)
    a2, F2 = s.get_state()
    alpha_new = alpha.copy()
    alpha_new[B] = aB
    assert np.array_equal(a2, alpha_new)
    Fref = oracle.responses(w.X, w.y, p, alpha_new)
    err = np.abs(F2 - Fref) / np.maximum(np.abs(Fref), 1.0)
    assert np.max(err) <= 1e-5, np.max(err)


@pytest.mark.parametrize("name,n,d", [("C1", 400, None), ("C2", 300, None)])
def test_pair_mode_follows_oracle_trajectory(name, n, d):
    # working_set = 2 performs exactly one maximal-violating-pair step per
    # outer iteration, so the first steps coincide with the oracle's
    w = _work(name, n, d)
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    N = oracle.num_vars(w.type, w.n)
    k = 20
    r = oracle.solve(w.X, w.y, p, np.zeros(N), np.zeros(w.n), max_steps=k)
    s = _solver(w, 2)
    it, gap = s.iterate(k)
    a, F = s.get_state()
    assert it == k
    np.testing.assert_allclose(a, r.alpha, rtol=1e-6, atol=1e-9 * w.C)
    np.testing.assert_allclose(F, r.F, rtol=1e-5, atol=1e-5)
