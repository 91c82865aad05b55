"""The CSR path on the GPU against the CPU oracle (which takes CSR input).

Kernel rows within 1e-5 relative; full training: dual objective within 1e-4
relative, the oracle's KKT gap of the GPU's alpha within tol, decision
values within 1e-3 absolute and labels at least 99.9% equal.  CSR and dense
copies of the same matrix give the same model to rounding (their dot
products are summed in different orders); the row cache changes no bits;
device (torch sparse CSR) and host input give the same bits; a malformed
matrix is refused by the device check.
"""
import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _c5(n, n_test=400):
    return workloads.make("C5", n=n, n_test=n_test)


def _c4_csr(n):
    w = workloads.make("C4", n=n, n_test=300)
    w.X, w.Xt = sp.csr_matrix(w.X), sp.csr_matrix(w.Xt)
    return w


def _ragged(n, d, seed):
    # rows of 0 to 40 nonzeros (empty rows included), N(0,1) values
    rng = np.random.default_rng(seed)
    nnz = rng.integers(0, 41, size=n)
    nnz[::17] = 0
    rows, cols = [], []
    for i, k in enumerate(nnz):
        rows.append(np.full(k, i))
        cols.append(np.sort(rng.choice(d, size=k, replace=False)))
    r = np.concatenate(rows)
    c = np.concatenate(cols)
    v = rng.standard_normal(r.size).astype(np.float32)
    X = sp.csr_matrix((v, (r, c)), shape=(n, d), dtype=np.float32)
    X.sort_indices()
    y = np.where(rng.standard_normal(n) + np.asarray(X.sum(axis=1)).ravel()
                 > 0, 1.0, -1.0).astype(np.float32)
    return X, y


@pytest.mark.parametrize("n,d,seed", [(333, 1000, 1), (1000, 97, 2),
                                      (130, 2000, 3)])
def test_kernel_rows_csr(n, d, seed):
    X, y = _ragged(n, d, seed)
    gamma = 0.05
    s = nv.Solver(X, y, type=C_SVC, C=1.0, gamma=gamma, tol=1e-3)
    rng = np.random.default_rng(n)
    idx = np.concatenate([[0, n - 1], rng.choice(n, 14, replace=False)])
    K = s.rows(idx)
    ref = oracle.kernel_rows(X, gamma, idx)
    err = np.abs(K - ref) - (1e-5 * np.abs(ref) + 1e-12)
    assert np.max(err) <= 0, np.max(np.abs(K - ref) / (np.abs(ref) + 1e-30))
    for j, i in enumerate(idx):
        assert K[j, i] == 1.0


def test_kernel_rows_csr_skewed_rows():
    # every 16th row holds 600 nonzeros, the others 1: padding the rows to
    # their slice's longest would pass 4 x nnz, so the row kernel walks the
    # CSR rows themselves (the other tests take the sliced copy)
    rng = np.random.default_rng(7)
    n, d = 160, 1000
    rows, cols = [], []
    for i in range(n):
        k = 600 if i % 16 == 0 else 1
        rows.append(np.full(k, i))
        cols.append(np.sort(rng.choice(d, size=k, replace=False)))
    r, c = np.concatenate(rows), np.concatenate(cols)
    v = (0.1 * rng.standard_normal(r.size)).astype(np.float32)
    X = sp.csr_matrix((v, (r, c)), shape=(n, d), dtype=np.float32)
    X.sort_indices()
    y = np.where(np.arange(n) % 2 == 0, 1.0, -1.0).astype(np.float32)
    gamma = 0.05
    s = nv.Solver(X, y, type=C_SVC, C=1.0, gamma=gamma, tol=1e-3)
    idx = np.array([0, 1, 16, 17, 31, 32, 63, 64, 100, 128, 144, 159,
                    2, 48, 80, 96])
    K = s.rows(idx)
    ref = oracle.kernel_rows(X, gamma, idx)
    err = np.abs(K - ref) - (1e-5 * np.abs(ref) + 1e-12)
    assert np.max(err) <= 0, np.max(np.abs(K - ref) / (np.abs(ref) + 1e-30))


def _check(w, m, ref, p):
    info = m.info()
    assert info["status"] == nv.SVM_OK
    idx, coef, alpha = nv.svm_model_get(m, 0, with_alpha=True)
    assert info["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)
    F = oracle.responses(w.X, w.y, p, alpha)
    summ = oracle.state_summary(w.y, p, alpha, F, w.d)
    assert summ.gap <= w.tol + 1e-5, summ.gap
    D = nv.svm_predict(m, w.Xt)
    Dref = oracle.model_decision(w.X, w.y, p, ref, w.Xt)
    assert np.max(np.abs(D - Dref)) <= 1e-3, np.max(np.abs(D - Dref))
    if w.type == C_SVC:
        L = nv.svm_predict_labels(m, w.Xt)
        assert np.mean(L == np.where(Dref >= 0, 1, -1)) >= 0.999


@pytest.mark.parametrize("n", [3000])
def test_train_c5_recipe_against_oracle(n):
    w = _c5(n)
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    ref = oracle.train(w.X, w.y, p)
    m = nv.svm_train(w.X, w.y, type=w.type, C=w.C, gamma=w.gamma, tol=w.tol)
    _check(w, m, ref, p)


def test_train_wide_ragged_csr_against_oracle():
    # d = 2000: more columns than the selection block has threads (its
    # column numbering takes the general scan), rows of 0 to 40 nonzeros
    from types import SimpleNamespace
    X, y = _ragged(1600, 2000, 7)
    w = SimpleNamespace(X=X[:1300], y=y[:1300], Xt=X[1300:], yt=y[1300:],
                        d=2000, type=C_SVC, C=1.0, eps=0.0, gamma=0.05,
                        tol=1e-3)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    ref = oracle.train(w.X, w.y, p)
    m = nv.svm_train(w.X, w.y, type=C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    _check(w, m, ref, p)


def test_train_svr_csr_against_oracle():
    w = workloads.make("C2", n=2000, n_test=300)
    w.X[np.abs(w.X) < 0.5] = 0.0  # about half the entries zero
    w.Xt[np.abs(w.Xt) < 0.5] = 0.0
    w.X, w.Xt = sp.csr_matrix(w.X), sp.csr_matrix(w.Xt)
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    ref = oracle.train(w.X, w.y, p)
    m = nv.svm_train(w.X, w.y, type=w.type, C=w.C, epsilon=w.eps,
                     gamma=w.gamma, tol=w.tol)
    _check(w, m, ref, p)


def test_ovr_c4_csr_against_oracle():
    w = _c4_csr(2000)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    refs = oracle.train_ovr(w.X, w.y, w.n_classes, p)
    m = nv.svm_train_ovr(w.X, w.y, w.n_classes, C=w.C, gamma=w.gamma,
                         tol=w.tol)
    for c in range(w.n_classes):
        assert m.info(c)["dual_obj"] == pytest.approx(refs[c].obj, rel=1e-4)
    D = nv.svm_predict(m, w.Xt)
    Dref = np.stack([oracle.model_decision(
        w.X, np.where(w.y == c, 1.0, -1.0).astype(np.float32), p, refs[c],
        w.Xt) for c in range(w.n_classes)], axis=1)
    assert np.max(np.abs(D - Dref)) <= 1e-3
    L = nv.svm_predict_labels(m, w.Xt)
    assert np.mean(L == np.argmax(Dref, axis=1)) >= 0.999


def test_sparse_decision_path_against_oracle():
    # ragged rows (0 to 40 nonzeros, some past the 32 the kernel holds in
    # registers) and three one-vs-rest outputs: a CSR model's predictions on
    # CSR rows go through the support rows by column; the oracle sums c K
    # directly over the GPU's support vectors
    X, _ = _ragged(1200, 500, 21)
    labels = np.random.default_rng(5).integers(0, 3, 1200).astype(np.int32)
    m = nv.svm_train_ovr(X, labels, 3, C=1.0, gamma=0.05, tol=1e-3)
    Xt, _ = _ragged(700, 500, 22)
    D = nv.svm_predict(m, Xt)
    for c in range(3):
        idx, coef, _ = nv.svm_model_get(m, c, with_alpha=True)
        SV = oracle.Matrix(X).rows(idx)
        Dsame = oracle.decision(SV, coef, m.info(c)["b"], Xt, 0.05)
        Kabs = oracle.decision(SV, np.abs(coef), 0.0, Xt, 0.05)
        assert np.max(np.abs(D[:, c] - Dsame) / (Kabs + 1.0)) <= 1e-6
    # empty query set, and a query set of only empty rows
    assert nv.svm_predict(m, sp.csr_matrix((0, 500), dtype=np.float32)
                          ).shape == (0, 3)
    Z = sp.csr_matrix((5, 500), dtype=np.float32)
    Dz = nv.svm_predict(m, Z)
    for c in range(3):
        idx, coef, _ = nv.svm_model_get(m, c)
        Dref = oracle.decision(oracle.Matrix(X).rows(idx), coef,
                               m.info(c)["b"], Z, 0.05)
        np.testing.assert_allclose(Dz[:, c], Dref, rtol=1e-6, atol=1e-9)


def test_csr_and_dense_give_the_same_model():
    X, y = _ragged(1500, 300, 7)
    kw = dict(type=C_SVC, C=1.0, gamma=0.02, tol=1e-3)
    mc = nv.svm_train(X, y, **kw)
    md = nv.svm_train(X.toarray(), y, **kw)
    # both stop within tol of the same optimum (their paths may differ)
    assert mc.info()["dual_obj"] == pytest.approx(md.info()["dual_obj"],
                                                  rel=1e-4)
    Dc = nv.svm_predict(mc, X)
    Dd = nv.svm_predict(md, X.toarray())
    assert np.max(np.abs(Dc - Dd)) <= 1e-3
    # CSR queries against a dense-trained model, and the reverse: the same
    # model, so only the order of the fp32 dot products differs
    assert np.max(np.abs(nv.svm_predict(md, X) - Dd)) <= 1e-4
    assert np.max(np.abs(nv.svm_predict(mc, X.toarray()) - Dc)) <= 1e-4


def test_csr_cache_changes_no_bits():
    w = _c5(4000)
    kw = dict(type=w.type, C=w.C, gamma=w.gamma, tol=w.tol)
    off = nv.svm_train(w.X, w.y, cache_bytes=-1, **kw)
    on = nv.svm_train(w.X, w.y, cache_bytes=0, **kw)
    a_off = nv.svm_model_get(off, 0, with_alpha=True)[2]
    a_on = nv.svm_model_get(on, 0, with_alpha=True)[2]
    np.testing.assert_array_equal(a_on, a_off)
    assert on.info()["dual_obj"] == off.info()["dual_obj"]
    assert on.info()["cache_hits"] > 0


def test_device_csr_input_matches_host():
    import torch
    w = _c5(2000)
    Xd = torch.sparse_csr_tensor(
        torch.from_numpy(w.X.indptr.astype(np.int64)),
        torch.from_numpy(w.X.indices.astype(np.int64)),
        torch.from_numpy(w.X.data.astype(np.float32)), size=w.X.shape,
        device="cuda")
    yd = torch.from_numpy(w.y).cuda()
    kw = dict(type=w.type, C=w.C, gamma=w.gamma, tol=w.tol)
    mh = nv.svm_train(w.X, w.y, **kw)
    md = nv.svm_train(Xd, yd, **kw)
    np.testing.assert_array_equal(nv.svm_model_get(md, 0, with_alpha=True)[2],
                                  nv.svm_model_get(mh, 0, with_alpha=True)[2])


@pytest.mark.parametrize("fault", ["unsorted", "repeat", "range", "ptr", "nan"])
def test_malformed_csr_is_refused(fault):
    X, y = _ragged(200, 50, 11)
    data, ind, ptr = X.data.copy(), X.indices.copy(), X.indptr.copy()
    row = int(np.argmax(np.diff(ptr) >= 3))
    a = ptr[row]
    if fault == "unsorted":
        ind[a], ind[a + 1] = ind[a + 1], ind[a]
    elif fault == "repeat":
        ind[a + 1] = ind[a]
    elif fault == "range":
        ind[a] = 50
    elif fault == "ptr":
        ptr[row + 1] = ptr[row] - 1
    else:
        data[a] = np.nan
    class Raw:  # CSR arrays as given, no checks on the host side
        pass
    bad = Raw()
    bad.data, bad.indices, bad.indptr, bad.shape = data, ind, ptr, X.shape
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(bad, y, type=C_SVC, C=1.0, gamma=0.1)
    assert e.value.status == nv.SVM_E_INVALID
