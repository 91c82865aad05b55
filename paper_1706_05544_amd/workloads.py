"""Seeded synthetic workloads for the kernel-SVM solver.

This module only draws random inputs; it holds none of the solver's
arithmetic.  Both the HIP path and the CPU oracle are fed from it.

The paper times its solver on two unnamed data sets (Section 5: eps-SVR on
113,978 x 120 and C-SVC on 68,971 x 501) that are not available here, so the
five synthetic problems below stand in for them.  Each is generated in fp64
with NumPy's PCG64, cast to fp32, then its rows are shuffled.  Seeds: the
training set of problem k uses 1000k + 1, its test set 1000k + 2 and any
shared structure (prototypes, weight vector) 1000k.

  C1  C-SVC   n=2000,   d=20,  x = y*0.5*1 + N(0,I), 1000 per class
  C2  eps-SVR n=20000,  d=50,  x ~ U[-1,1], z = sin(3x0) + 0.5 x1 x2 + N(0,0.1^2)
  C3  C-SVC   n=100000, d=128, x = y*0.2*1 + N(0,I), 50000 per class
  C4  10-class one-vs-rest, n=500000, d=784, sparse prototypes (~20% nnz)
  C5  C-SVC   n=2e6,    d=1000, CSR, 20 distinct columns per row, N(0,1)
      values, y = sign(w.x + N(0,0.5^2)) with sign(0) = +1

C3B is C3 with the class means at +-0.1133*1 (10 % Bayes error instead of
1.2 %; the same seeds): the same bytes per iteration, more iterations and
support vectors.

Two more take the shapes of the paper's own data sets, with the C2 and C3
recipes (the paper gives no value distributions), and 10 % more points as
the test set:

  PSVR  eps-SVR n=113978, d=120, the C2 recipe (the target uses x0, x1, x2;
        the other 117 features are U[-1,1] noise), gamma = 1/120
  PSVC  C-SVC   n=68971,  d=501, the C3 recipe (means +-0.2*1), gamma = 1/501

Sizes can be overridden (``n=``, ``n_test=``) to get a smaller problem with
the same recipe; the data then differ from the full-size draw.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

C_SVC = 0
EPS_SVR = 1


@dataclass
class Workload:
    name: str
    type: int                  # C_SVC or EPS_SVR
    X: object                  # fp32 (n, d) ndarray or scipy CSR matrix
    y: np.ndarray              # fp32 labels +-1 / targets; int32 classes (OvR)
    Xt: object
    yt: np.ndarray
    C: float
    gamma: float
    eps: float = 0.1
    tol: float = 1e-3
    n_classes: int = 2
    meta: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return self.X.shape[0]

    @property
    def d(self) -> int:
        return self.X.shape[1]


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _gauss_pair(k: int, n: int, n_test: int, d: int, shift: float,
                C: float, gamma: float, name: str) -> Workload:
    """Two isotropic Gaussians N(+-shift*1, I), equal class sizes."""
    rng = _rng(1000 * k + 1)
    y = np.concatenate([np.ones(n // 2), -np.ones(n - n // 2)])
    X = y[:, None] * shift + rng.standard_normal((n, d))
    perm = rng.permutation(n)
    X, y = X[perm], y[perm]
    rt = _rng(1000 * k + 2)
    yt = np.where(rt.random(n_test) < 0.5, 1.0, -1.0)
    Xt = yt[:, None] * shift + rt.standard_normal((n_test, d))
    return Workload(name, C_SVC, X.astype(np.float32), y.astype(np.float32),
                    Xt.astype(np.float32), yt.astype(np.float32), C=C,
                    gamma=gamma)


def c1(n: int = 2000, n_test: int = 1000) -> Workload:
    return _gauss_pair(1, n, n_test, 20, 0.5, 1.0, 1.0 / 20, "C1")


def c2(n: int = 20000, n_test: int = 5000, d: int = 50, k: int = 2,
       name: str = "C2") -> Workload:

    def draw(rng, m):
        X = rng.uniform(-1.0, 1.0, (m, d))
        z = (np.sin(3.0 * X[:, 0]) + 0.5 * X[:, 1] * X[:, 2]
             + rng.normal(0.0, 0.1, m))
        return X, z

    rng = _rng(1000 * k + 1)
    X, z = draw(rng, n)
    perm = rng.permutation(n)
    X, z = X[perm], z[perm]
    Xt, zt = draw(_rng(1000 * k + 2), n_test)
    return Workload(name, EPS_SVR, X.astype(np.float32), z.astype(np.float32),
                    Xt.astype(np.float32), zt.astype(np.float32), C=10.0,
                    gamma=1.0 / d, eps=0.1)


def c3(n: int = 100000, n_test: int = 20000) -> Workload:
    return _gauss_pair(3, n, n_test, 128, 0.2, 1.0, 1.0 / 128, "C3")


def c3b(n: int = 100000, n_test: int = 20000) -> Workload:
    # C3's draw at the offset that gives a 10 % Bayes error:
    # Phi(-0.1133 sqrt(128)) = 0.10
    return _gauss_pair(3, n, n_test, 128, 0.1133, 1.0, 1.0 / 128, "C3B")


def psvr(n: int = 113978, n_test: int = 11398) -> Workload:
    return c2(n, n_test, d=120, k=6, name="PSVR")


def psvc(n: int = 68971, n_test: int = 6897) -> Workload:
    return _gauss_pair(7, n, n_test, 501, 0.2, 1.0, 1.0 / 501, "PSVC")


def _c4_prototypes(d: int, n_classes: int, support: int):
    rng = _rng(4000)
    sup = np.stack([rng.choice(d, support, replace=False)
                    for _ in range(n_classes)])
    inten = rng.uniform(0.0, 1.0, (n_classes, support))
    return sup, inten


def _c4_draw(rng, m, labels, d, sup, inten, extra):
    X = np.zeros((m, d))
    support = sup.shape[1]
    for c in range(sup.shape[0]):
        rows = np.nonzero(labels == c)[0]
        if len(rows) == 0:
            continue
        k = len(rows)
        keep = rng.random((k, support)) >= 0.1          # 10% dropout
        vals = inten[c][None, :] + rng.normal(0.0, 0.1, (k, support))
        vals = np.clip(vals, 0.0, 1.0) * keep
        X[np.ix_(rows, sup[c])] = vals
        off = np.setdiff1d(np.arange(d), sup[c])
        # 16 off-support pixels per sample set to U[0,1]
        pick = np.argsort(rng.random((k, len(off))), axis=1)[:, :extra]
        X[rows[:, None], off[pick]] = rng.uniform(0.0, 1.0, (k, extra))
    return X


def c4(n: int = 500000, n_test: int = 50000, layout: str = "dense") -> Workload:
    d, n_classes, support, extra = 784, 10, 157, 16
    sup, inten = _c4_prototypes(d, n_classes, support)
    rng = _rng(4001)
    labels = np.repeat(np.arange(n_classes), n // n_classes)
    labels = np.concatenate([labels, np.arange(n - len(labels))])
    X = _c4_draw(rng, n, labels, d, sup, inten, extra)
    perm = rng.permutation(n)
    X, labels = X[perm], labels[perm]
    rt = _rng(4002)
    lt = rt.integers(0, n_classes, n_test)
    Xt = _c4_draw(rt, n_test, lt, d, sup, inten, extra)
    X = X.astype(np.float32)
    Xt = Xt.astype(np.float32)
    if layout == "csr":
        import scipy.sparse as sp
        X, Xt = sp.csr_matrix(X), sp.csr_matrix(Xt)
    return Workload("C4", C_SVC, X, labels.astype(np.int32), Xt,
                    lt.astype(np.int32), C=10.0, gamma=0.02,
                    n_classes=n_classes)


def _c5_draw(rng, m, d, nnz, w):
    import scipy.sparse as sp
    cols = np.sort(rng.integers(0, d, (m, nnz)), axis=1)
    while True:  # redraw rows with a repeated column
        bad = np.nonzero((np.diff(cols, axis=1) == 0).any(axis=1))[0]
        if len(bad) == 0:
            break
        cols[bad] = np.sort(rng.integers(0, d, (len(bad), nnz)), axis=1)
    vals = rng.standard_normal((m, nnz))
    score = (vals * w[cols]).sum(axis=1) + rng.normal(0.0, 0.5, m)
    y = np.where(score >= 0.0, 1.0, -1.0)
    indptr = np.arange(0, m * nnz + 1, nnz, dtype=np.int64)
    X = sp.csr_matrix((vals.reshape(-1).astype(np.float32),
                       cols.reshape(-1).astype(np.int32), indptr),
                      shape=(m, d))
    return X, y


def c5(n: int = 2000000, n_test: int = 1000000) -> Workload:
    d, nnz = 1000, 20
    w = _rng(5000).standard_normal(d)
    rng = _rng(5001)
    X, y = _c5_draw(rng, n, d, nnz, w)
    perm = rng.permutation(n)
    X, y = X[perm], y[perm]
    Xt, yt = _c5_draw(_rng(5002), n_test, d, nnz, w)
    return Workload("C5", C_SVC, X, y.astype(np.float32), Xt,
                    yt.astype(np.float32), C=1.0, gamma=0.05)


def make(name: str, n: Optional[int] = None, n_test: Optional[int] = None,
         **kw) -> Workload:
    gen = {"C1": c1, "C2": c2, "C3": c3, "C3B": c3b, "C4": c4, "C5": c5,
           "PSVR": psvr, "PSVC": psvc}[name.upper().replace("-", "")]
    args = dict(kw)
    if n is not None:
        args["n"] = n
    if n_test is not None:
        args["n_test"] = n_test
    return gen(**args)


def tiny(n: int, d: int, seed: int, kind: str = "svc",
         duplicates: bool = False):
    """Small random problems for brute-force checks."""
    rng = _rng(seed)
    X = rng.standard_normal((n, d))
    if duplicates and n >= 3:
        X[2] = X[0]
    if kind == "svc":
        y = np.where(rng.random(n) < 0.5, 1.0, -1.0)
        y[0], y[1] = 1.0, -1.0
    else:
        y = np.sin(2.0 * X[:, 0]) + 0.3 * rng.standard_normal(n)
    return X.astype(np.float32), y.astype(np.float32)
