"""Scaling, k-fold cross-validation and tuning on the GPU against the oracle.

The GPU trains a fold on the whole feature store with the held-out rows
outside both index sets; the oracle trains on the subset itself (the plain
definition).  Bars as elsewhere: decision values within 1e-3 absolute (in
the units of the scaled problem), labels at least 99.9 % equal, dual
objective within 1e-4 relative; the metrics the library reports equal the
metrics of the decision values it returned, and agree with the oracle's to
within the rows whose label differs.
"""
import numpy as np
import pytest
import scipy.sparse as sp

import oracle
from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _skewed(n, seed, n_test=1000):
    rng = np.random.default_rng(seed)
    sc = np.array([1, 10, 0.01, 100, 1, 1, 3, 0.5])
    off = np.array([0, 5, -3, 1000, 0, 0, 1, -1])

    def draw(m):
        G = rng.standard_normal((m, 8))
        X = G * sc + off
        X[:, 4] = 2.5
        y = np.where(G[:, 0] + G[:, 1] - G[:, 2] + G[:, 6] +
                     0.5 * rng.standard_normal(m) > 0.3, 1.0, -1.0)
        return X.astype(np.float32), y.astype(np.float32)
    X, y = draw(n)
    Xt, yt = draw(n_test)
    return X, y, Xt, yt


def test_scaled_train_svc():
    X, y, Xt, _ = _skewed(1500, 1)
    p = Params(C_SVC, C=1.0, gamma=0.125, tol=1e-3)
    ref, _ = oracle.train_scaled(X, y, p, Xt)
    m = nv.svm_train(X, y, C=1.0, gamma=0.125, tol=1e-3, scale=1)
    assert m.info()["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)
    # decision values and labels at tol 1e-5 on both sides: on this problem
    # the oracle's own D moves by 1.1e-3 between tol 1e-3 and 1e-6
    p5 = Params(C_SVC, C=1.0, gamma=0.125, tol=1e-5)
    _, Dref = oracle.train_scaled(X, y, p5, Xt)
    m5 = nv.svm_train(X, y, C=1.0, gamma=0.125, tol=1e-5, scale=1)
    D = nv.svm_predict(m5, Xt)
    assert np.max(np.abs(D - Dref)) <= 1e-3
    L = nv.svm_predict_labels(m5, Xt)
    assert np.mean(L == np.where(Dref >= 0, 1, -1)) >= 0.999
    # the same data unscaled is a different (badly conditioned) problem
    m0 = nv.svm_train(X, y, C=1.0, gamma=0.125, tol=1e-3)
    assert m0.info()["dual_obj"] != pytest.approx(ref.obj, rel=1e-2)


def test_scaled_train_svr_targets_in_their_units():
    w = workloads.c2(n=1500, n_test=500)
    z, zt = w.y * 3.0 + 1.0, w.yt * 3.0 + 1.0
    p = Params(EPS_SVR, C=w.C, eps=w.eps, gamma=w.gamma, tol=1e-3)
    ref, Dref = oracle.train_scaled(w.X, z, p, w.Xt)
    m = nv.svm_train(w.X, z, type=EPS_SVR, C=w.C, epsilon=w.eps,
                     gamma=w.gamma, tol=1e-3, scale=1)
    assert m.info()["dual_obj"] == pytest.approx(ref.obj, rel=1e-4)
    D = nv.svm_predict(m, w.Xt)
    (_,), (sd,) = oracle.scale_stats(np.asarray(z)[:, None])
    assert np.max(np.abs(D - Dref)) <= 1e-3 * sd
    assert np.mean((D - zt) ** 2) < 0.5 * np.var(zt)  # it learnt something


def _gpu_metrics_match(stats, D, type_, y=None, labels=None):
    m = oracle.metrics(type_, D, y, labels)
    for k, v in m.items():
        assert stats[k] == pytest.approx(v, rel=1e-9, abs=1e-12), k


def test_cv_svc():
    w = workloads.c1(n=1500, n_test=10)
    k = 5
    fold = np.random.default_rng(7).integers(0, k, w.n)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    Dref = oracle.cross_validate(w.X, w.y, p, k, fold)
    D, st = nv.svm_cross_validate(w.X, w.y, k=k, fold=fold, C=w.C,
                                  gamma=w.gamma, tol=w.tol)
    assert st["rc"] == nv.SVM_OK and st["folds"] == k and st["n"] == w.n
    assert np.max(np.abs(D - Dref)) <= 1e-3
    assert np.mean(np.sign(D + 1e-300) == np.sign(Dref + 1e-300)) >= 0.999
    _gpu_metrics_match(st, D, C_SVC, w.y)
    ref = oracle.metrics(C_SVC, Dref, w.y)
    assert abs(st["accuracy"] - ref["accuracy"]) <= 2.0 / w.n


def test_cv_fold_equals_training_on_its_rows():
    # the held-out rows outside I_up and I_low: the fold's model is the model
    # of the other rows, trained on them alone
    w = workloads.c1(n=1200, n_test=10)
    k = 3
    fold = np.arange(w.n) % k
    D, _ = nv.svm_cross_validate(w.X, w.y, k=k, fold=fold, C=w.C,
                                 gamma=w.gamma, tol=w.tol)
    for f in range(k):
        tr, te = fold != f, fold == f
        m = nv.svm_train(w.X[tr], w.y[tr], C=w.C, gamma=w.gamma, tol=w.tol)
        Df = nv.svm_predict(m, w.X[te])
        assert np.max(np.abs(D[te] - Df)) <= 1e-9, np.max(np.abs(D[te] - Df))


def test_cv_svr_scaled():
    w = workloads.c2(n=1200, n_test=10)
    z = w.y * 2.0 - 0.5
    k = 4
    p = Params(EPS_SVR, C=w.C, eps=w.eps, gamma=w.gamma, tol=w.tol)
    # the oracle's equivalent: standardise all rows once, cross-validate,
    # map the decision values back to the units of the targets
    mu, sd = oracle.scale_stats(w.X)
    Xs = oracle.scale_apply(w.X, mu, sd)
    (zm,), (zs,) = oracle.scale_stats(np.asarray(z)[:, None])
    zsc = oracle.scale_apply(np.asarray(z)[:, None], np.array([zm]),
                             np.array([zs]))[:, 0]
    Dref = oracle.cross_validate(Xs, zsc, p, k) * zs + zm
    D, st = nv.svm_cross_validate(w.X, z, k=k, type=EPS_SVR, C=w.C,
                                  epsilon=w.eps, gamma=w.gamma, tol=w.tol,
                                  scale=1)
    assert np.max(np.abs(D - Dref)) <= 1e-3 * zs
    _gpu_metrics_match(st, D, EPS_SVR, z)
    ref = oracle.metrics(EPS_SVR, Dref, z)
    assert st["mse"] == pytest.approx(ref["mse"], rel=1e-3)
    assert st["scc"] == pytest.approx(ref["scc"], rel=1e-3)


def test_cv_ovr():
    w = workloads.make("C4", n=1200, n_test=10)
    k = 3
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    Dref = oracle.cross_validate(w.X, None, p, k, labels=w.y,
                                 n_classes=w.n_classes)
    D, st = nv.svm_cross_validate(w.X, labels=w.y, n_classes=w.n_classes,
                                  k=k, C=w.C, gamma=w.gamma, tol=w.tol)
    assert D.shape == (w.n, w.n_classes)
    assert np.max(np.abs(D - Dref)) <= 1e-3
    assert np.mean(D.argmax(1) == Dref.argmax(1)) >= 0.999
    _gpu_metrics_match(st, D, C_SVC, labels=w.y)


def test_cv_csr():
    w = workloads.make("C5", n=2000, n_test=10)
    k = 3
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    Dref = oracle.cross_validate(w.X, w.y, p, k)
    D, st = nv.svm_cross_validate(w.X, w.y, k=k, C=w.C, gamma=w.gamma,
                                  tol=w.tol)
    assert np.max(np.abs(D - Dref)) <= 1e-3
    _gpu_metrics_match(st, D, C_SVC, w.y)


def test_tune_grid():
    w = workloads.c1(n=800, n_test=10)
    k = 3
    Cs = np.array([0.01, 0.1, 1.0, 10.0, 1.0, 10.0])
    gs = np.array([0.05, 0.05, 0.05, 0.05, 0.5, 0.5])
    err, best = nv.svm_tune(w.X, w.y, k=k, C=Cs, gamma=gs, tol=w.tol)
    ref = []
    for C, g in zip(Cs, gs):
        D = oracle.cross_validate(w.X, w.y, Params(C_SVC, C=C, gamma=g,
                                                   tol=w.tol), k)
        ref.append(oracle.metrics(C_SVC, D, w.y)["error"])
    ref = np.array(ref)
    np.testing.assert_allclose(err, ref, atol=2.0 / w.n)
    assert best == int(np.argmin(err))
    assert err[best] <= ref.min() + 2.0 / w.n


def test_cv_device_features_same_as_host():
    import torch
    w = workloads.c1(n=900, n_test=10)
    D, st = nv.svm_cross_validate(w.X, w.y, k=3, C=w.C, gamma=w.gamma,
                                  tol=w.tol)
    Dd, std = nv.svm_cross_validate(torch.from_numpy(w.X).to("cuda:0"), w.y,
                                    k=3, C=w.C, gamma=w.gamma, tol=w.tol)
    np.testing.assert_array_equal(D, Dd)
    assert st["accuracy"] == std["accuracy"] and st["iters"] == std["iters"]
