"""Lockstep trainings (one-vs-rest classes, cross-validation folds) on the GPU.

Problems in lockstep share the selection launch and the pass over X, but
each problem's kernel values, F updates and candidates are computed as for
that problem alone: its iterations, alpha and bias are the bits of the same
training run on its own without the row cache (which lockstep does not
use).  So the bar here is bitwise equality with the sequential trainings
(cache off), which the other GPU tests tie to the oracle; one test also
compares a lockstep cross-validation with the oracle's directly (decision
values within 1e-3, labels at least 99.9 % equal).  Cases: group sizes 2
to 4 and a last group of one, a group that shrinks as its problems finish
at different iterations, C-SVC, eps-SVR, a polynomial kernel, one-vs-rest
with its classes in lockstep, 784 features (two problems fit the LDS),
ragged row counts.
"""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, EPS_SVR, POLY, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _same_ovr(m1, m2, n_classes):
    for c in range(n_classes):
        i1, c1, a1 = nv.svm_model_get(m1, c, with_alpha=True)
        i2, c2, a2 = nv.svm_model_get(m2, c, with_alpha=True)
        np.testing.assert_array_equal(a1, a2)
        np.testing.assert_array_equal(i1, i2)
        np.testing.assert_array_equal(c1, c2)
        f1, f2 = m1.info(c), m2.info(c)
        for k in ("iters", "b", "dual_obj", "gap", "kernel_rows", "status"):
            assert f1[k] == f2[k], (c, k, f1[k], f2[k])


@pytest.mark.parametrize("lockstep", [2, 4])
def test_ovr_lockstep_equals_sequential(lockstep):
    # 784 features: at most two problems per pass; lockstep = 4 is clamped
    w = workloads.make("C4", n=1531, n_test=300)
    kw = dict(C=w.C, gamma=w.gamma, tol=w.tol, cache_bytes=-1)
    seq = nv.svm_train_ovr(w.X, w.y, w.n_classes, **kw)
    lock = nv.svm_train_ovr(w.X, w.y, w.n_classes, lockstep=lockstep, **kw)
    _same_ovr(seq, lock, w.n_classes)
    iters = [seq.info(c)["iters"] for c in range(w.n_classes)]
    assert len(set(iters)) > 1  # the groups shrink as classes finish
    np.testing.assert_array_equal(nv.svm_predict(seq, w.Xt),
                                  nv.svm_predict(lock, w.Xt))


def test_ovr_lockstep_few_features_four_problems():
    # 10 classes in groups of 4, 4 and 2; 40 features: four problems a pass
    X, lab = _ten_classes()
    k = 10
    kw = dict(C=2.0, gamma=0.02, tol=1e-3, cache_bytes=-1)
    seq = nv.svm_train_ovr(X, lab, k, **kw)
    lock = nv.svm_train_ovr(X, lab, k, lockstep=4, **kw)
    _same_ovr(seq, lock, k)


@pytest.mark.parametrize("k,lockstep", [(5, 4), (3, 3), (4, 2)])
def test_cv_svc_lockstep_equals_sequential(k, lockstep):
    w = workloads.c1(n=1501, n_test=10)
    fold = np.random.default_rng(k).integers(0, k, w.n)
    kw = dict(k=k, fold=fold, C=w.C, gamma=w.gamma, tol=w.tol,
              cache_bytes=-1)
    D0, s0 = nv.svm_cross_validate(w.X, w.y, **kw)
    D1, s1 = nv.svm_cross_validate(w.X, w.y, lockstep=lockstep, **kw)
    np.testing.assert_array_equal(D0, D1)
    for key in ("iters", "kernel_rows", "accuracy", "status"):
        assert s0[key] == s1[key], key


def test_cv_svr_lockstep_equals_sequential():
    w = workloads.c2(n=1203, n_test=10)
    kw = dict(k=4, type=EPS_SVR, C=w.C, epsilon=w.eps, gamma=w.gamma,
              tol=w.tol, cache_bytes=-1)
    D0, s0 = nv.svm_cross_validate(w.X, w.y, **kw)
    D1, s1 = nv.svm_cross_validate(w.X, w.y, lockstep=4, **kw)
    np.testing.assert_array_equal(D0, D1)
    assert s0["iters"] == s1["iters"] and s0["mse"] == s1["mse"]


def test_cv_poly_scaled_lockstep_equals_sequential():
    w = workloads.c1(n=1200, n_test=10)
    kw = dict(k=3, C=w.C, gamma=0.05, kernel=POLY, degree=3, coef0=1.0,
              tol=w.tol, cache_bytes=-1, scale=1)
    D0, s0 = nv.svm_cross_validate(w.X, w.y, **kw)
    D1, s1 = nv.svm_cross_validate(w.X, w.y, lockstep=3, **kw)
    np.testing.assert_array_equal(D0, D1)
    assert s0["iters"] == s1["iters"]


def test_cv_ovr_lockstep_equals_sequential():
    # (fold, class) trainings in groups: 2 folds x 10 classes, two a pass
    w = workloads.make("C4", n=1200, n_test=10)
    kw = dict(labels=w.y, n_classes=w.n_classes, k=2, C=w.C, gamma=w.gamma,
              tol=w.tol, cache_bytes=-1)
    D0, s0 = nv.svm_cross_validate(w.X, **kw)
    D1, s1 = nv.svm_cross_validate(w.X, lockstep=2, **kw)
    np.testing.assert_array_equal(D0, D1)
    assert s0["iters"] == s1["iters"]


def test_cv_lockstep_against_oracle():
    w = workloads.c1(n=1500, n_test=10)
    k = 4
    fold = np.random.default_rng(9).integers(0, k, w.n)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    Dref = oracle.cross_validate(w.X, w.y, p, k, fold)
    D, st = nv.svm_cross_validate(w.X, w.y, k=k, fold=fold, C=w.C,
                                  gamma=w.gamma, tol=w.tol, lockstep=4)
    assert st["rc"] == nv.SVM_OK
    assert np.max(np.abs(D - Dref)) <= 1e-3
    assert np.mean(np.sign(D + 1e-300) == np.sign(Dref + 1e-300)) >= 0.999


def test_tune_lockstep_equals_sequential():
    # 3 grid points x 3 folds in groups of 4: groups mix grid points with
    # different C and gamma
    w = workloads.c1(n=900, n_test=10)
    Cs = np.array([0.1, 1.0, 10.0])
    gs = np.array([0.05, 0.05, 0.2])
    kw = dict(k=3, C=Cs, gamma=gs, tol=w.tol, cache_bytes=-1)
    e0, b0 = nv.svm_tune(w.X, w.y, **kw)
    e1, b1 = nv.svm_tune(w.X, w.y, lockstep=4, **kw)
    np.testing.assert_array_equal(e0, e1)
    assert b0 == b1


def test_tune_svr_epsilon_grid_lockstep():
    w = workloads.c2(n=800, n_test=10)
    eps = np.array([0.05, 0.1, 0.3])
    kw = dict(k=2, type=EPS_SVR, C=np.full(3, w.C), gamma=np.full(3, w.gamma),
              epsilon=eps, tol=w.tol, cache_bytes=-1)
    e0, b0 = nv.svm_tune(w.X, w.y, **kw)
    e1, b1 = nv.svm_tune(w.X, w.y, lockstep=4, **kw)
    np.testing.assert_array_equal(e0, e1)
    assert b0 == b1


def _ten_classes(n=2003, d=40, seed=11):
    rng = np.random.default_rng(seed)
    P = rng.standard_normal((10, d)) * 1.5
    lab = rng.integers(0, 10, n).astype(np.int32)
    X = (P[lab] + rng.standard_normal((n, d))).astype(np.float32)
    return X, lab


def test_lockstep_iteration_cap():
    # max_iter between the classes' iteration counts: some classes stop at
    # the cap (warning) while the others of their group converge; the same
    # states as one class after another
    X, lab = _ten_classes()
    kw = dict(C=2.0, gamma=0.02, tol=1e-3, cache_bytes=-1)
    free = nv.svm_train_ovr(X, lab, 10, **kw)
    its = sorted(free.info(c)["iters"] for c in range(10))
    cap = its[5]
    assert its[0] < cap < its[-1]
    seq = nv.svm_train_ovr(X, lab, 10, max_iter=cap, **kw)
    lock = nv.svm_train_ovr(X, lab, 10, max_iter=cap, lockstep=4, **kw)
    _same_ovr(seq, lock, 10)
    st = [lock.info(c)["status"] for c in range(10)]
    assert nv.SVM_W_MAX_ITER in st and nv.SVM_OK in st


def test_lockstep_profile_splits_the_pass():
    # with profiling, each launch's time and shared bytes are split over its
    # problems: the per-training launches add up to the passes of the group
    w = workloads.c1(n=1500, n_test=10)
    kw = dict(k=4, C=w.C, gamma=w.gamma, tol=w.tol, cache_bytes=-1,
              profile=1)
    _, s0 = nv.svm_cross_validate(w.X, w.y, **kw)
    _, s1 = nv.svm_cross_validate(w.X, w.y, lockstep=4, **kw)
    assert s1["row_kernel_launches"] == s0["row_kernel_launches"]
    assert s1["row_kernel_ms"] > 0
    # X is read once per pass instead of once per problem
    assert s1["row_kernel_bytes"] < s0["row_kernel_bytes"]


def test_fullsize_c3_cv10_lockstep4():
    # the configuration `bench.py --cv 10 --lockstep 4` times: C3 at full
    # size (n = 100000, d = 128), 10 folds in groups of 4, 4 and 2
    w = workloads.make("C3")
    kw = dict(k=10, C=w.C, gamma=w.gamma, tol=w.tol, cache_bytes=-1)
    D0, s0 = nv.svm_cross_validate(w.X, w.y, **kw)
    D1, s1 = nv.svm_cross_validate(w.X, w.y, lockstep=4, **kw)
    np.testing.assert_array_equal(D0, D1)
    assert s0["iters"] == s1["iters"] and s0["accuracy"] == s1["accuracy"]
    assert s1["rc"] == nv.SVM_OK and 0.98 < s1["accuracy"] < 1.0


@pytest.mark.parametrize("d", [900, 2000])
def test_lockstep_many_features(d):
    # d = 900: two problems fill the LDS of a pass; d = 2000: not even two
    # fit, so the folds run one after another (without the cache)
    rng = np.random.default_rng(d)
    n = 603
    y = np.where(rng.standard_normal(n) > 0, 1.0, -1.0).astype(np.float32)
    X = (rng.standard_normal((n, d)) + 0.05 * y[:, None]).astype(np.float32)
    kw = dict(k=3, C=1.0, gamma=1.0 / d, tol=1e-3, cache_bytes=-1)
    D0, s0 = nv.svm_cross_validate(X, y, **kw)
    D1, s1 = nv.svm_cross_validate(X, y, lockstep=4, **kw)
    np.testing.assert_array_equal(D0, D1)
    assert s0["iters"] == s1["iters"] and s1["rc"] == nv.SVM_OK
