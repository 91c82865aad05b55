"""The factored sparse decision path on the GPU against the oracle.

A CSR model whose support rows are sparse predicts CSR rows through the
support rows split into chunks by column: the constant term of the pairs
that share no column, and the dot products of the pairs that do.  The
oracle sums c_j K(sv_j, x) directly in fp64 over the GPU model's support
vectors, so each case isolates the prediction (within 1e-6 of
sum_j |c_j K| + 1, the bound of fp32 kernel values summed in fp64).

Cases: several chunks (more than 2048 support rows), query rows longer
than one wave (more than 64 nonzeros) and with more than 16 passes of
entries against one chunk, empty query rows, one and three outputs, rows
whose norm is too large for the factored form (the direct formula), the
polynomial, sigmoid and linear kernels, the table path (still built on
request) against it, the same bits on a second call, and the recompute of F after training
(K(x_i, x_i) = 1 for a training row's own support row).
"""
import os

import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from paper_1706_05544_amd import native as nv

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, scope="module")
def _factored_path():
    # The library takes the factored path for rows that share fewer than 0.3
    # columns with a support row on average; these tests take it whatever
    # the shape (the developer switch), so that every case below runs it.
    os.environ["SVM_SPARSE_PATH"] = "factor"
    yield
    os.environ.pop("SVM_SPARSE_PATH", None)


def _rows(n, d, nz_max, seed, long_rows=0, long_nz=150, scale_rows=0):
    """CSR rows with 0..nz_max nonzeros at uniform columns, N(0,1) values;
    some rows with long_nz nonzeros, some scaled by 10."""
    rng = np.random.default_rng(seed)
    nnz = rng.integers(0, nz_max + 1, size=n)
    nnz[::23] = 0
    if long_rows:
        nnz[1:1 + long_rows] = long_nz
    rows, cols = [], []
    for i, k in enumerate(nnz):
        rows.append(np.full(k, i))
        cols.append(np.sort(rng.choice(d, size=k, replace=False)))
    r = np.concatenate(rows)
    c = np.concatenate(cols)
    v = rng.standard_normal(r.size).astype(np.float32)
    X = sp.csr_matrix((v, (r, c)), shape=(n, d), dtype=np.float32)
    X.sort_indices()
    if scale_rows:
        X = sp.diags(np.where(np.arange(n) < n - scale_rows, 1.0, 10.0)
                     .astype(np.float32)) @ X
        X = sp.csr_matrix(X, dtype=np.float32)
        X.sort_indices()
    return X


def _check(m, X, Xt, D, gamma, kind=oracle.RBF, degree=3, coef0=0.0):
    D = D.reshape(Xt.shape[0], -1)
    for c in range(D.shape[1]):
        idx, coef, _ = nv.svm_model_get(m, c, with_alpha=True)
        SV = oracle.Matrix(X).rows(idx)
        b = m.info(c)["b"]
        ref = oracle.decision(SV, coef, b, Xt, gamma, 0, kind, degree, coef0)
        Kabs = oracle.decision(SV, np.abs(coef), 0.0, Xt, gamma, 0, kind,
                               degree, coef0)
        if kind != oracle.RBF:
            # |K| of a kernel of the dot product, summed with |c|
            Kt = np.abs(oracle.kernel(SV, Xt, gamma, kind, degree, coef0))
            Kabs = Kt.T @ np.abs(coef)
        err = np.max(np.abs(D[:, c] - ref) / (Kabs + 1.0))
        assert err <= 1e-6, (c, err)
    return D


@pytest.fixture(scope="module")
def big_model():
    # about 4000 support rows (random labels): two chunks
    X = _rows(6000, 800, 30, 1)
    y = np.where(np.random.default_rng(2).standard_normal(6000) > 0, 1.0,
                 -1.0).astype(np.float32)
    m = nv.svm_train(X, y, C=1.0, gamma=0.05, tol=1e-3)
    assert m.info()["n_sv_output"] > 2048
    return X, m


def test_chunks_long_rows_and_empty_rows(big_model):
    X, m = big_model
    Xt = _rows(500, 800, 30, 3, long_rows=6, long_nz=700)
    D = nv.svm_predict(m, Xt)
    _check(m, X, Xt, D, 0.05)
    # the same bits on a second call
    assert np.array_equal(nv.svm_predict(m, Xt), D)
    # only empty rows: e^0 C0 + b
    Z = sp.csr_matrix((7, 800), dtype=np.float32)
    _check(m, X, Z, nv.svm_predict(m, Z), 0.05)


def test_rows_too_large_for_the_factored_form(big_model):
    X, m = big_model
    # rows scaled by 10: gamma log2(e) |x|^2 is far above the bound, so
    # these rows take the direct formula
    Xt = _rows(300, 800, 30, 4, scale_rows=100)
    _check(m, X, Xt, nv.svm_predict(m, Xt), 0.05)


def test_table_path_still_serves_and_agrees(big_model):
    # SVM_SPARSE_PATH=table builds a model without the chunks by column, so
    # it predicts through the table path; the two trainings differ only in
    # how the final responses were recomputed (each within tol)
    X, m = big_model
    Xt = _rows(400, 800, 30, 5, long_rows=3)
    D = nv.svm_predict(m, Xt)
    os.environ["SVM_SPARSE_PATH"] = "table"
    try:
        y = np.where(np.random.default_rng(2).standard_normal(6000) > 0,
                     1.0, -1.0).astype(np.float32)
        m2 = nv.svm_train(X, y, C=1.0, gamma=0.05, tol=1e-3)
    finally:
        os.environ["SVM_SPARSE_PATH"] = "factor"
    D2 = _check(m2, X, Xt, nv.svm_predict(m2, Xt), 0.05)
    assert m2.info()["dual_obj"] == pytest.approx(m.info()["dual_obj"],
                                                  rel=1e-6)
    assert np.max(np.abs(D - D2[:, 0])) <= 1e-3


def test_three_outputs():
    X = _rows(2500, 600, 25, 6)
    labels = np.random.default_rng(7).integers(0, 3, 2500).astype(np.int32)
    m = nv.svm_train_ovr(X, labels, 3, C=1.0, gamma=0.05, tol=1e-3)
    Xt = _rows(400, 600, 25, 8, long_rows=2, long_nz=90)
    _check(m, X, Xt, nv.svm_predict(m, Xt), 0.05)


@pytest.mark.parametrize("kind,degree,coef0,gamma", [
    (oracle.POLY, 3, 1.0, 0.1), (oracle.SIGMOID, 3, 0.0, 0.05),
    (oracle.LINEAR, 3, 0.0, 1.0)])
def test_other_kernels(kind, degree, coef0, gamma):
    X = _rows(1500, 700, 20, 9)
    y = np.where(np.random.default_rng(10).standard_normal(1500) > 0, 1.0,
                 -1.0).astype(np.float32)
    m = nv.svm_train(X, y, C=1.0, gamma=gamma, tol=1e-3, kernel=kind,
                     degree=degree, coef0=coef0, max_iter=20000)
    Xt = _rows(300, 700, 20, 11)
    _check(m, X, Xt, nv.svm_predict(m, Xt), gamma, kind, degree, coef0)


def test_recompute_after_training_matches_oracle_responses():
    # the responses the solver recomputes from alpha (K(x_i, x_i) = 1 for
    # a row's own support row) give the oracle's gap and bias
    X = _rows(3000, 900, 20, 12)
    y = np.where(np.random.default_rng(13).standard_normal(3000) > 0, 1.0,
                 -1.0).astype(np.float32)
    s = nv.Solver(X, y, C=1.0, gamma=0.05, tol=1e-3)
    p = oracle.Params(oracle.C_SVC, C=1.0, gamma=0.05, tol=1e-3)
    r = oracle.solve(X, y, p, np.zeros(3000), np.zeros(3000), max_steps=200)
    s.set_state(r.alpha, np.zeros(3000))
    gap, b, obj, status = s.finish(max_passes=0)
    Fo = oracle.responses(X, y, p, r.alpha)
    ref = oracle.state_summary(y, p, r.alpha, Fo, d=900)
    _, F = s.get_state()
    c = y * r.alpha
    Kabs = oracle.decision(X, np.abs(c), 0.0, X, 0.05)
    assert np.max(np.abs(F - Fo) / (Kabs + 1.0)) <= 1e-6
    assert gap == pytest.approx(ref.gap, abs=1e-5)
    assert b == pytest.approx(ref.b, abs=1e-5)
