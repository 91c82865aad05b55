"""End-to-end training and prediction on the GPU against the CPU oracle.

Bars (from the parity contract): dual objective within 1e-4 relative,
decision values within 1e-3 absolute, labels at least 99.9% equal; the
constraints hold and the KKT gap, recomputed by the oracle from the GPU's
alpha, is within tol.  Prediction alone is checked on the GPU's own model
against the oracle's direct fp64 sum (1e-6 relative to the sum of |c K|).
"""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _train_both(w, **kw):
    p = Params(w.type, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    ref = oracle.train(w.X, w.y, p)
    m = nv.svm_train(w.X, w.y, type=w.type, C=w.C, epsilon=w.eps,
                     gamma=w.gamma, tol=w.tol, **kw)
    return p, ref, m


def _check_model(w, p, ref, m, test_rows=True):
    info = m.info()
    assert info["status"] == nv.SVM_OK
    idx, coef, alpha = nv.svm_model_get(m, 0, with_alpha=True)
    N = oracle.num_vars(w.type, w.n)
    assert alpha.shape == (N,)
    # constraints
    assert np.all(alpha >= 0) and np.all(alpha <= w.C)
    yy = (np.where(w.y > 0, 1.0, -1.0) if w.type == C_SVC
          else np.concatenate([np.ones(w.n), -np.ones(w.n)]))
    assert abs(yy @ alpha) <= 1e-9 * w.C * N
    # KKT gap of the GPU's alpha, recomputed by the oracle in fp64
    F = oracle.responses(w.X, w.y, p, alpha)
    summ = oracle.state_summary(w.y, p, alpha, F, w.d)
    assert summ.gap <= w.tol + 1e-5, summ.gap
    # objective
    assert info["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)
    assert summ.obj == pytest.approx(info["dual_obj"], rel=1e-7)
    assert info["b"] == pytest.approx(summ.b, abs=2e-4)
    # model arrays agree with alpha
    c = oracle.coefficients(w.type, w.n, w.y, alpha)
    assert list(idx) == list(np.nonzero(c)[0])
    np.testing.assert_array_equal(coef, c[idx])
    # prediction on held-out points
    X2 = w.Xt if test_rows else w.X
    D = nv.svm_predict(m, X2)
    Dref = oracle.model_decision(w.X, w.y, p, ref, X2)
    assert np.max(np.abs(D - Dref)) <= 1e-3, np.max(np.abs(D - Dref))
    if w.type == C_SVC:
        L = nv.svm_predict_labels(m, X2)
        Lref = np.where(Dref >= 0, 1, -1)
        assert np.mean(L == Lref) >= 0.999
    # prediction alone: the GPU model through the oracle's direct sum
    Dsame = oracle.decision(w.X[idx], coef, info["b"], X2, w.gamma)
    Kabs = oracle.decision(w.X[idx], np.abs(coef), 0.0, X2, w.gamma)
    assert np.max(np.abs(D - Dsame) / (Kabs + 1.0)) <= 1e-6
    return info


def test_c1_full():
    w = workloads.c1()
    p, ref, m = _train_both(w)
    info = _check_model(w, p, ref, m)
    assert info["iters"] > 0 and info["kernel_rows"] > 0


def test_c2_svr_subsample():
    w = workloads.c2(n=3000, n_test=1000)
    p, ref, m = _train_both(w)
    _check_model(w, p, ref, m)


def test_c3_subsample():
    w = workloads.c3(n=6000, n_test=2000)
    p, ref, m = _train_both(w)
    _check_model(w, p, ref, m)


@pytest.mark.parametrize("q", [2, 4, 32, 64])
def test_other_working_set_sizes(q):
    w = workloads.c1(n=700, n_test=300)
    p, ref, m = _train_both(w, working_set=q)
    _check_model(w, p, ref, m)


def test_device_inputs_match_host_inputs():
    import torch
    w = workloads.c1(n=500, n_test=200)
    mh = nv.svm_train(w.X, w.y, C=w.C, gamma=w.gamma)
    md = nv.svm_train(torch.from_numpy(w.X).cuda(),
                      torch.from_numpy(w.y).cuda(), C=w.C, gamma=w.gamma)
    ah = nv.svm_model_get(mh, 0, with_alpha=True)[2]
    ad = nv.svm_model_get(md, 0, with_alpha=True)[2]
    assert np.array_equal(ah, ad)
    Dh = nv.svm_predict(mh, w.Xt)
    Dd = nv.svm_predict(md, torch.from_numpy(w.Xt).cuda()).cpu().numpy()
    assert np.array_equal(Dh, Dd)


def test_runs_are_bitwise_repeatable():
    w = workloads.c2(n=800, n_test=100)
    a = [nv.svm_model_get(nv.svm_train(w.X, w.y, type=w.type, C=w.C,
                                       epsilon=w.eps, gamma=w.gamma),
                          0, with_alpha=True)[2] for _ in range(2)]
    assert np.array_equal(a[0], a[1])


def test_edge_two_points_and_duplicates():
    X = np.array([[0.0, 0.0], [1.0, 0.5]], np.float32)
    y = np.array([1.0, -1.0], np.float32)
    m = nv.svm_train(X, y, C=10.0, gamma=0.5, tol=1e-6)
    info = m.info()
    k = np.exp(-0.5 * 1.25)
    assert info["dual_obj"] == pytest.approx(-1.0 / (1 - k), rel=1e-6)
    Xd, yd = workloads.tiny(9, 3, 7, "svc", duplicates=True)
    yd[2] = -yd[0]
    p = Params(C_SVC, C=1.0, gamma=0.5, tol=1e-3)
    ref = oracle.train(Xd, yd, p)
    md = nv.svm_train(Xd, yd, C=1.0, gamma=0.5)
    assert md.info()["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)


def test_edge_max_iter_and_empty_predict():
    w = workloads.c1(n=400, n_test=10)
    m = nv.svm_train(w.X, w.y, max_iter=3, C=w.C, gamma=w.gamma)
    assert m.status == nv.SVM_W_MAX_ITER
    info = m.info()
    assert info["status"] == nv.SVM_W_MAX_ITER and info["iters"] == 3
    assert info["gap"] > w.tol
    D = nv.svm_predict(m, np.zeros((0, w.d), np.float32))
    assert D.shape == (0,)


def test_edge_d1_and_ragged_features():
    # a tight tol: with d = 1 the kernel matrix is badly conditioned and two
    # tol-1e-3 stopping points give decision values ~2e-3 apart
    for d in (1, 5, 17):
        w = workloads.c1(n=257, n_test=33)
        X = np.ascontiguousarray(w.X[:, :d])
        Xt = np.ascontiguousarray(w.Xt[:, :d])
        p = Params(C_SVC, C=1.0, gamma=1.0 / d, tol=1e-5)
        ref = oracle.train(X, w.y, p)
        m = nv.svm_train(X, w.y, C=1.0, gamma=1.0 / d, tol=1e-5)
        assert m.info()["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)
        D = nv.svm_predict(m, Xt)
        Dref = oracle.model_decision(X, w.y, p, ref, Xt)
        assert np.max(np.abs(D - Dref)) <= 1e-3


def test_wrong_feature_count_in_predict():
    w = workloads.c1(n=100, n_test=10)
    m = nv.svm_train(w.X, w.y)
    with pytest.raises(nv.SvmError) as e:
        nv.svm_predict(m, w.Xt[:, :5])
    assert e.value.status == nv.SVM_E_INVALID
