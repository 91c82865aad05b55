"""Oracle pins for scaling, k-fold cross-validation, metrics and tuning.

Section 3 lists, among the features of the interface: scaling of the
training data, K-fold cross validation, tuning of C, eps and the kernel
parameters, and accuracy / correlation / mean squared error.  The oracle
takes e1071's definitions: each feature standardised with its mean and
sample standard deviation (constant columns left as they are; eps-SVR
targets too), each row predicted by the model trained on the other folds.
Pinned by: scipy's z-score, scikit-learn's cross_val_predict with LIBSVM on
the same folds (endpoint slack at tol 1e-3), scikit-learn's and scipy's
metrics, and invariants.
"""
import numpy as np
import pytest
from scipy.stats import pearsonr, zscore
from sklearn.metrics import accuracy_score, mean_squared_error
from sklearn.model_selection import PredefinedSplit, cross_val_predict
from sklearn.svm import SVC, SVR

from oracle import C_SVC, EPS_SVR, Params
from paper_1706_05544_amd import workloads


def _skewed(n, seed):
    # features of very different scales and offsets, one constant column
    rng = np.random.default_rng(seed)
    G = rng.standard_normal((n, 6))
    X = G * np.array([1, 10, 0.01, 100, 1, 1]) + np.array([0, 5, -3, 1000, 0, 0])
    X[:, 4] = 2.5
    y = np.where(G[:, 0] + G[:, 1] - G[:, 2] + 0.5 * rng.standard_normal(n)
                 > 0.3, 1.0, -1.0)
    assert 0.2 < np.mean(y > 0) < 0.8  # both classes, well mixed
    return X.astype(np.float32), y.astype(np.float32)


def test_scale_stats_match_zscore(orc):
    X, _ = _skewed(300, 1)
    mu, sd = orc.scale_stats(X)
    assert sd[4] == 0.0 and mu[4] == 2.5
    Xs = orc.scale_apply(X, mu, sd)
    cols = [0, 1, 2, 3, 5]
    ref = zscore(X[:, cols].astype(np.float64), axis=0, ddof=1)
    np.testing.assert_allclose(Xs[:, cols], ref, rtol=1e-6, atol=1e-6)
    np.testing.assert_array_equal(Xs[:, 4], X[:, 4])  # constant: as given
    np.testing.assert_allclose(Xs[:, cols].astype(np.float64).mean(axis=0),
                               0.0, atol=1e-6)
    np.testing.assert_allclose(Xs[:, cols].astype(np.float64).std(axis=0,
                                                                  ddof=1),
                               1.0, rtol=1e-6)


def test_metrics_match_sklearn(orc):
    rng = np.random.default_rng(2)
    y = np.where(rng.standard_normal(200) > 0, 1.0, -1.0)
    D = y * 0.5 + rng.standard_normal(200)
    m = orc.metrics(C_SVC, D, y)
    assert m["accuracy"] == pytest.approx(
        accuracy_score(y, np.where(D >= 0, 1.0, -1.0)), abs=1e-15)
    z = rng.standard_normal(200)
    Dz = z + 0.3 * rng.standard_normal(200)
    m = orc.metrics(EPS_SVR, Dz, z)
    assert m["mse"] == pytest.approx(mean_squared_error(z, Dz), rel=1e-12)
    assert m["scc"] == pytest.approx(pearsonr(Dz, z)[0] ** 2, rel=1e-10)
    lab = rng.integers(0, 4, 200)
    D4 = rng.standard_normal((200, 4))
    D4[np.arange(200), lab] += 1.0
    m = orc.metrics(C_SVC, D4, labels=lab)
    assert m["accuracy"] == pytest.approx(np.mean(D4.argmax(1) == lab))


def test_cv_svc_matches_libsvm_folds(orc):
    w = workloads.c1(n=600, n_test=10)
    k = 5
    fold = np.random.default_rng(3).integers(0, k, w.n)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=1e-3)
    D = orc.cross_validate(w.X, w.y, p, k, fold)
    lib = SVC(C=w.C, kernel="rbf", gamma=w.gamma, tol=1e-3, shrinking=False)
    Dl = cross_val_predict(lib, w.X.astype(np.float64), w.y,
                           cv=PredefinedSplit(fold),
                           method="decision_function")
    np.testing.assert_allclose(D, Dl, atol=2e-3)
    assert np.mean(np.sign(D) == np.sign(Dl)) >= 0.995
    # each fold's model never saw its rows: training on everything differs
    r = orc.train(w.X, w.y, p)
    Dall = orc.model_decision(w.X, w.y, p, r, w.X)
    assert np.max(np.abs(Dall - D)) > 1e-2


def test_cv_svr_matches_libsvm_folds(orc):
    w = workloads.c2(n=500, n_test=10)
    k = 4
    p = Params(EPS_SVR, C=w.C, eps=w.eps, gamma=w.gamma, tol=1e-3)
    D = orc.cross_validate(w.X, w.y, p, k)
    fold = np.arange(w.n) % k
    lib = SVR(C=w.C, epsilon=w.eps, kernel="rbf", gamma=w.gamma, tol=1e-3,
              shrinking=False)
    Dl = cross_val_predict(lib, w.X.astype(np.float64),
                           w.y.astype(np.float64), cv=PredefinedSplit(fold))
    np.testing.assert_allclose(D, Dl, atol=3e-3)


def test_scaled_training_invariant_to_feature_affine_maps(orc):
    # standardisation removes per-feature offsets and positive scales: the
    # same problem up to the fp32 rounding of the scaled values
    X, y = _skewed(300, 4)
    rng = np.random.default_rng(5)
    Xt = X[:50]
    a = rng.uniform(0.5, 4.0, X.shape[1]).astype(np.float32)
    c = rng.uniform(-10, 10, X.shape[1]).astype(np.float32)
    p = Params(C_SVC, C=1.0, gamma=0.2, tol=1e-6)
    r1, D1 = orc.train_scaled(X, y, p, Xt)
    r2, D2 = orc.train_scaled(X * a + c, y, p, Xt * a + c)
    assert r1.obj == pytest.approx(r2.obj, rel=1e-4)
    np.testing.assert_allclose(D1, D2, atol=1e-3)


def test_scaled_svr_targets_back_in_their_units(orc):
    w = workloads.c2(n=400, n_test=100)
    p = Params(EPS_SVR, C=w.C, eps=0.05, gamma=w.gamma, tol=1e-4)
    _, D = orc.train_scaled(w.X, w.y * 100 + 7, p, w.Xt)
    # the model fits targets of mean 7 and scale 100: its error is ~100x
    # the unscaled problem's
    mse = np.mean((D - (w.yt * 100 + 7)) ** 2)
    assert 100 < mse < 1e5
    assert abs(np.mean(D) - 7) < 30


def test_tuning_error_is_cv_error(orc):
    w = workloads.c1(n=300, n_test=10)
    k = 3
    errs = []
    for C in (0.01, 1.0, 100.0):
        p = Params(C_SVC, C=C, gamma=w.gamma, tol=1e-3)
        D = orc.cross_validate(w.X, w.y, p, k)
        errs.append(orc.metrics(C_SVC, D, w.y)["error"])
    # a very small C underfits this mixture
    assert errs[0] > min(errs)
