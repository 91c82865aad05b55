"""The seeded input generators: shapes, parameters, determinism and the
recipe of each workload (small sizes; the full-size draws follow the same
code)."""
import numpy as np
import pytest
import scipy.sparse as sp

from paper_1706_05544_amd import workloads as wl


@pytest.mark.parametrize("name,d,typ,gamma", [
    ("C1", 20, wl.C_SVC, 1 / 20), ("C2", 50, wl.EPS_SVR, 1 / 50),
    ("C3", 128, wl.C_SVC, 1 / 128), ("C3B", 128, wl.C_SVC, 1 / 128),
    ("PSVR", 120, wl.EPS_SVR, 1 / 120),
    ("PSVC", 501, wl.C_SVC, 1 / 501)])
def test_dense_shapes_and_parameters(name, d, typ, gamma):
    w = wl.make(name, n=300, n_test=40)
    assert w.X.shape == (300, d) and w.Xt.shape == (40, d)
    assert w.X.dtype == np.float32 and w.y.dtype == np.float32
    assert w.type == typ and w.gamma == pytest.approx(gamma)
    if typ == wl.C_SVC:
        assert set(np.unique(w.y)) <= {-1.0, 1.0}
        assert (w.y > 0).sum() == 150  # equal class sizes, shuffled
    else:
        assert np.all(np.abs(w.X) <= 1.0)  # U[-1, 1] features
    again = wl.make(name, n=300, n_test=40)
    assert np.array_equal(w.X, again.X) and np.array_equal(w.yt, again.yt)


def test_full_size_defaults():
    # the sizes of the data sets of Section 5 (not drawn: only the
    # generators' defaults are read)
    import inspect
    assert inspect.signature(wl.psvr).parameters["n"].default == 113978
    assert inspect.signature(wl.psvc).parameters["n"].default == 68971


def test_names_are_case_and_dash_insensitive():
    a = wl.make("p-svr", n=50, n_test=5)
    b = wl.make("PSVR", n=50, n_test=5)
    assert a.name == "PSVR" and np.array_equal(a.X, b.X)


def test_c2_recipe_target():
    # z = sin(3 x0) + 0.5 x1 x2 + N(0, 0.1^2): the residual has sd 0.1
    w = wl.c2(n=4000, n_test=10)
    X = w.X.astype(np.float64)
    r = w.y - (np.sin(3 * X[:, 0]) + 0.5 * X[:, 1] * X[:, 2])
    assert abs(r.mean()) < 0.01 and 0.09 < r.std() < 0.11
    # the same recipe at d = 120 with its own seeds
    p = wl.psvr(n=4000, n_test=10)
    Xp = p.X.astype(np.float64)
    rp = p.y - (np.sin(3 * Xp[:, 0]) + 0.5 * Xp[:, 1] * Xp[:, 2])
    assert 0.09 < rp.std() < 0.11
    assert not np.array_equal(p.X[:, :50], w.X)


def test_gaussian_pair_means():
    # x = y * 0.2 * 1 + N(0, I): the class means sit at +-0.2
    w = wl.psvc(n=4000, n_test=10)
    X = w.X.astype(np.float64)
    m_pos = X[w.y > 0].mean()
    m_neg = X[w.y < 0].mean()
    assert abs(m_pos - 0.2) < 0.01 and abs(m_neg + 0.2) < 0.01


def test_c3b_is_c3_at_a_smaller_offset():
    # the same seeds: the noise is C3's, the means move from 0.2 to 0.1133
    a = wl.c3(n=1000, n_test=10)
    b = wl.c3b(n=1000, n_test=10)
    assert np.array_equal(a.y, b.y)
    diff = (a.X.astype(np.float64) - b.X) * a.y[:, None]
    assert np.allclose(diff, 0.2 - 0.1133, atol=1e-6)


def test_c5_rows_have_twenty_distinct_sorted_columns():
    w = wl.c5(n=2000, n_test=100)
    assert sp.isspmatrix_csr(w.X) and w.X.shape == (2000, 1000)
    nnz = np.diff(w.X.indptr)
    assert np.all(nnz == 20)
    cols = w.X.indices.reshape(2000, 20)
    assert np.all(np.diff(cols, axis=1) > 0)


def test_c4_one_vs_rest_labels():
    w = wl.c4(n=500, n_test=50)
    assert w.n_classes == 10 and w.y.dtype == np.int32
    assert np.bincount(w.y, minlength=10).tolist() == [50] * 10
    assert np.all((w.X >= 0) & (w.X <= 1))
    c = wl.c4(n=500, n_test=50, layout="csr")
    assert sp.isspmatrix_csr(c.X)
    assert np.array_equal(c.X.toarray(), w.X)
