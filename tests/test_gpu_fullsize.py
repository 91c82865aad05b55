"""Parity at the full sizes of the workloads, in the launch configuration of
a training run (the library picks the row kernel's grid and tiles from n
and d; the test hooks launch the same kernels on the same grid).

Per step, from identical states reached by the oracle (maximal-violating-
pair steps from alpha = 0): kernel rows over all n (1e-5 relative), the
working set and the gap (exact), and the response update over all n (1e-5
relative to max(|F|, 1)).

Whole trainings, where the oracle cannot run a whole training in a test:
properties that hold at any size, checked by the oracle on the GPU's
result: the box and equality constraints; the KKT gap of the GPU's alpha
over every training row (C2, C3; for C4's 10 classes over 500000 rows, on
2000 sampled rows a class: a subset's gap is at most the whole's, so this
one is a necessary check only), with the responses summed by the oracle in
fp64,
within tol plus the fp32 kernel's 1e-5 relative bound over the sum of
|c_j K_ij|; the dual objective recomputed by the oracle from the GPU's
alpha (only the variables with alpha != 0 contribute), within the bound
that 1e-5 relative on every kernel value gives; decision values on
sampled test points against the oracle's direct fp64 sum over the GPU's
support vectors (1e-6 relative to the sum of |c K|).
"""
import copy

import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu

_cache = {}


def _full(key):
    """Full-size workload: C2, C3, C4 (dense), C4csr, C5."""
    if key not in _cache:
        if key == "C4csr":
            w = copy.copy(_full("C4"))
            w.X, w.Xt = sp.csr_matrix(w.X), sp.csr_matrix(w.Xt)
        else:
            w = workloads.make(key)
        _cache[key] = w
    return _cache[key]


def _binary(w):
    """Labels of the binary problem (C4: class 0 against the rest)."""
    if w.n_classes > 2:
        return np.where(w.y == 0, 1.0, -1.0).astype(np.float32)
    return w.y


def _rows(X, idx):
    return oracle.Matrix(X).rows(idx)


def _params(w):
    return Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)


def _solver(w, y):
    return nv.Solver(w.X, y, type=w.type, C=w.C, epsilon=w.eps,
                     gamma=w.gamma, tol=w.tol)


KEYS = ["C2", "C3", "C4", "C4csr", "C5"]


@pytest.mark.parametrize("key", KEYS)
def test_full_kernel_rows(key):
    w = _full(key)
    s = _solver(w, _binary(w))
    n = w.n
    rng = np.random.default_rng(7)
    idx = np.concatenate([[0, n - 1], rng.choice(n, 14, replace=False)])
    K = s.rows(idx)
    ref = oracle.kernel_rows(w.X, w.gamma, idx)
    err = np.abs(K - ref) - (1e-5 * np.abs(ref) + 1e-12)
    assert np.max(err) <= 0, np.max(np.abs(K - ref) / (np.abs(ref) + 1e-30))
    for j, i in enumerate(idx):
        assert K[j, i] == 1.0


@pytest.mark.parametrize("key", KEYS)
def test_full_select_and_update(key):
    w = _full(key)
    y = _binary(w)
    p = _params(w)
    N = oracle.num_vars(w.type, w.n)
    r = oracle.solve(w.X, y, p, np.zeros(N), np.zeros(w.n), max_steps=24)
    s = _solver(w, y)
    s.set_state(r.alpha, r.F)
    B, m, M = s.select()
    Be, me, Me = oracle.select(y, p, r.alpha, r.F, 16, d=w.d)
    assert m == me and M == Me
    assert list(B) == list(Be)
    itol = max(0.3 * (m - M), 0.5 * w.tol)
    aB, _ = oracle.subproblem(w.X, y, p, r.alpha, r.F, B, itol, 128)
    s.apply(B, aB)
    a2, F2 = s.get_state()
    alpha_new = r.alpha.copy()
    alpha_new[B] = aB
    assert np.array_equal(a2, alpha_new)
    c = oracle.coefficients(w.type, w.n, y, alpha_new)
    sv = np.nonzero(c)[0]
    Fref = oracle.decision(_rows(w.X, sv), c[sv], 0.0, w.X, w.gamma)
    err = np.abs(F2 - Fref) / np.maximum(np.abs(Fref), 1.0)
    assert np.max(err) <= 1e-5, np.max(err)


def _check_solution(w, y, p, m, output, n_sample=None, seed=11):
    """Constraints, KKT gap (over all rows, or n_sample sampled rows),
    objective and sampled predictions of one output of a trained model, all
    recomputed by the oracle."""
    info = m.info(output)
    assert info["status"] == nv.SVM_OK
    idx, coef, alpha = nv.svm_model_get(m, output, with_alpha=True)
    n, N = w.n, oracle.num_vars(w.type, w.n)
    assert alpha.shape == (N,)
    assert np.all(alpha >= 0) and np.all(alpha <= w.C)
    yy = (np.where(y > 0, 1.0, -1.0) if w.type == C_SVC
          else np.concatenate([np.ones(n), -np.ones(n)]))
    assert abs(yy @ alpha) <= 1e-9 * w.C * N
    c = oracle.coefficients(w.type, n, y, alpha)
    assert list(idx) == list(np.nonzero(c)[0])
    np.testing.assert_array_equal(coef, c[idx])
    SV = _rows(w.X, idx)

    def sub(rows):  # the variables of a subset of the samples
        if w.type == EPS_SVR:
            return np.concatenate([alpha[rows], alpha[n + rows]])
        return alpha[rows]

    # KKT gap over every row, or on a sample (a subset's gap is at most the
    # whole's)
    if n_sample is None:
        S = np.arange(n)
    else:
        rng = np.random.default_rng(seed)
        S = np.sort(rng.choice(n, min(n_sample, n), replace=False))
    XS = _rows(w.X, S)
    FS = oracle.decision(SV, coef, 0.0, XS, w.gamma)
    KS = oracle.decision(SV, np.abs(coef), 0.0, XS, w.gamma)
    summ = oracle.state_summary(y[S], p, sub(S), FS, w.d)
    assert summ.gap <= w.tol + 1e-5 * (np.max(KS) + 1.0), summ.gap
    # dual objective: only the variables with alpha != 0 contribute; the
    # GPU sums fp32 kernel values (1e-5 relative each), so the two differ by
    # at most 1e-5 / 2 |c|^T K |c|
    Fsv = oracle.decision(SV, coef, 0.0, SV, w.gamma)
    Ksv = oracle.decision(SV, np.abs(coef), 0.0, SV, w.gamma)
    obj = oracle.state_summary(y[idx], p, sub(idx), Fsv, w.d).obj
    bound = 0.5e-5 * (np.abs(coef) @ Ksv)
    assert abs(info["dual_obj"] - obj) <= bound, (info["dual_obj"], obj)
    return idx, coef, info


def _check_predict(w, m, outputs, n_sample=300, seed=13):
    D = nv.svm_predict(m, w.Xt)
    if D.ndim == 1:
        D = D[:, None]
    rng = np.random.default_rng(seed)
    T = np.sort(rng.choice(w.Xt.shape[0], n_sample, replace=False))
    XT = _rows(w.Xt, T)
    for o, (idx, coef, info) in enumerate(outputs):
        SV = _rows(w.X, idx)
        Dsame = oracle.decision(SV, coef, info["b"], XT, w.gamma)
        Kabs = oracle.decision(SV, np.abs(coef), 0.0, XT, w.gamma)
        assert np.max(np.abs(D[T, o] - Dsame) / (Kabs + 1.0)) <= 1e-6
    return D


@pytest.mark.parametrize("key", ["C2", "C3"])
def test_full_training(key):
    w = _full(key)
    p = _params(w)
    m = nv.svm_train(w.X, w.y, type=w.type, C=w.C, epsilon=w.eps,
                     gamma=w.gamma, tol=w.tol)
    out = _check_solution(w, w.y, p, m, 0)
    D = _check_predict(w, m, [out])
    if w.type == C_SVC:
        L = nv.svm_predict_labels(m, w.Xt)
        assert np.array_equal(L, np.where(D[:, 0] >= 0, 1, -1))


@pytest.mark.parametrize("key", ["C4", "C4csr"])
def test_full_training_ovr(key):
    w = _full(key)
    p = _params(w)
    m = nv.svm_train_ovr(w.X, w.y, w.n_classes, C=w.C, gamma=w.gamma,
                         tol=w.tol)
    assert m.n_outputs == w.n_classes
    outs = []
    for c in range(w.n_classes):
        yc = np.where(w.y == c, 1.0, -1.0).astype(np.float32)
        outs.append(_check_solution(w, yc, p, m, c, n_sample=2000, seed=c))
    D = _check_predict(w, m, outs)
    L = nv.svm_predict_labels(m, w.Xt)
    assert np.array_equal(L, np.argmax(D, axis=1))
