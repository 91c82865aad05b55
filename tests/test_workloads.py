"""Seeded generators: determinism, shapes and the stated structure."""
import numpy as np

from paper_1706_05544_amd import workloads


def test_deterministic_and_shapes():
    a = workloads.c1()
    b = workloads.c1()
    assert np.array_equal(a.X, b.X) and np.array_equal(a.y, b.y)
    assert a.X.shape == (2000, 20) and a.X.dtype == np.float32
    assert a.Xt.shape == (1000, 20)
    assert np.sum(a.y == 1) == 1000 and np.sum(a.y == -1) == 1000
    assert a.gamma == 1.0 / 20 and a.C == 1.0


def test_class_means_c3_small():
    w = workloads.c3(n=20000, n_test=100)
    assert w.X.shape == (20000, 128)
    mp = w.X[w.y > 0].mean()
    mn = w.X[w.y < 0].mean()
    assert abs(mp - 0.2) < 0.01 and abs(mn + 0.2) < 0.01


def test_c2_targets():
    w = workloads.c2(n=3000, n_test=100)
    assert w.type == workloads.EPS_SVR
    assert w.X.min() >= -1 and w.X.max() <= 1
    resid = w.y - (np.sin(3 * w.X[:, 0]) + 0.5 * w.X[:, 1] * w.X[:, 2])
    assert abs(np.std(resid) - 0.1) < 0.01


def test_c4_density_and_classes():
    w = workloads.c4(n=2000, n_test=200)
    dens = np.count_nonzero(w.X) / w.X.size
    assert 0.15 < dens < 0.25
    assert set(np.unique(w.y)) == set(range(10))
    assert w.X.min() >= 0 and w.X.max() <= 1


def test_c5_structure():
    w = workloads.c5(n=5000, n_test=100)
    X = w.X
    assert X.shape == (5000, 1000)
    assert np.all(np.diff(X.indptr) == 20)
    for i in range(0, 5000, 97):
        cols = X.indices[X.indptr[i]:X.indptr[i + 1]]
        assert np.all(np.diff(cols) > 0)
    assert set(np.unique(w.y)) == {-1.0, 1.0}
