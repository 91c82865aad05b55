"""CPU fp64 oracle for the kernel-SVM dual solve (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never does, and
the two share no code: this module is argument marshalling (ctypes) around
``svm_oracle.c``, which computes everything in fp64 from the paper's
statement of the problem (Wang et al., arXiv 1706.05544, Section 3, Eq. 1
and Eq. 2; maximal-violating-pair SMO as in LIBSVM, Chang & Lin 2011).

Parity pins: see the header of ``svm_oracle.c``.
"""
from __future__ import annotations

import ctypes as ct
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "svm_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

C_SVC = 0
EPS_SVR = 1
# kernels (Section 3's list, e1071 parameterisation)
LINEAR = 0
POLY = 1
RBF = 2
SIGMOID = 3


def build(force: bool = True) -> str:
    """Compile svm_oracle.c with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


class _Mat(ct.Structure):
    _fields_ = [("n", ct.c_int64), ("d", ct.c_int64), ("csr", ct.c_int32),
                ("val", ct.c_void_p), ("ld", ct.c_int64),
                ("row_ptr", ct.c_void_p), ("col", ct.c_void_p)]


class _Params(ct.Structure):
    _fields_ = [("type", ct.c_int32), ("C", ct.c_double), ("eps", ct.c_double),
                ("gamma", ct.c_double), ("tol", ct.c_double),
                ("max_iter", ct.c_int64), ("threads", ct.c_int32),
                ("kernel", ct.c_int32), ("degree", ct.c_int32),
                ("coef0", ct.c_double)]


class _Result(ct.Structure):
    _fields_ = [("iters", ct.c_int64), ("gap", ct.c_double), ("m", ct.c_double),
                ("M", ct.c_double), ("b", ct.c_double), ("obj", ct.c_double),
                ("n_sv", ct.c_int64), ("n_free", ct.c_int64),
                ("status", ct.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ct.CDLL(_LIB)
        P = ct.POINTER
        lib.orc_kernel.argtypes = [P(_Mat), P(_Mat), P(_Params), ct.c_void_p]
        lib.orc_kernel_rows.argtypes = [P(_Mat), P(_Params), ct.c_void_p,
                                        ct.c_int64, ct.c_int32, ct.c_void_p]
        lib.orc_num_vars.restype = ct.c_int64
        lib.orc_num_vars.argtypes = [ct.c_int32, ct.c_int64]
        lib.orc_solve.argtypes = [P(_Mat), ct.c_void_p, P(_Params), ct.c_int64,
                                  ct.c_void_p, ct.c_void_p, P(_Result)]
        lib.orc_train.argtypes = [P(_Mat), ct.c_void_p, P(_Params),
                                  ct.c_void_p, ct.c_void_p, P(_Result)]
        lib.orc_state_summary.argtypes = [ct.c_int64, ct.c_void_p, P(_Params),
                                          ct.c_void_p, ct.c_void_p, P(_Result)]
        lib.orc_responses.argtypes = [P(_Mat), ct.c_void_p, P(_Params),
                                      ct.c_void_p, ct.c_void_p]
        lib.orc_select.argtypes = [ct.c_int64, ct.c_void_p, P(_Params),
                                   ct.c_void_p, ct.c_void_p, ct.c_int32,
                                   ct.c_void_p, P(ct.c_int32),
                                   P(ct.c_double), P(ct.c_double)]
        lib.orc_subproblem.argtypes = [ct.c_int64, ct.c_void_p, P(_Params),
                                       ct.c_int32, ct.c_void_p, ct.c_void_p,
                                       ct.c_void_p, ct.c_void_p, ct.c_double,
                                       ct.c_int32, ct.c_void_p, P(ct.c_int32)]
        lib.orc_decision.argtypes = [P(_Mat), ct.c_void_p, ct.c_double,
                                     P(_Mat), P(_Params), ct.c_int32,
                                     ct.c_void_p]
        _lib = lib
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ct.c_void_p) if a is not None else None


class Matrix:
    """A dense fp32 row-major matrix or a CSR matrix (scipy-style arrays)."""

    def __init__(self, X):
        if hasattr(X, "indptr"):
            self.csr = True
            self.data = np.ascontiguousarray(X.data, dtype=np.float32)
            self.indptr = np.ascontiguousarray(X.indptr, dtype=np.int64)
            self.indices = np.ascontiguousarray(X.indices, dtype=np.int32)
            self.n, self.d = X.shape
            self.ld = 0
        else:
            self.csr = False
            self.data = np.ascontiguousarray(X, dtype=np.float32)
            assert self.data.ndim == 2
            self.n, self.d = self.data.shape
            self.ld = self.d
            self.indptr = self.indices = None
        self.s = _Mat(self.n, self.d, 1 if self.csr else 0, _ptr(self.data),
                      self.ld, _ptr(self.indptr), _ptr(self.indices))

    def rows(self, idx) -> "Matrix":
        idx = np.asarray(idx, dtype=np.int64)
        if not self.csr:
            return Matrix(self.data[idx])
        import scipy.sparse as sp
        m = sp.csr_matrix((self.data, self.indices, self.indptr),
                          shape=(self.n, self.d))
        return Matrix(m[idx])


def _as_mat(X) -> Matrix:
    return X if isinstance(X, Matrix) else Matrix(X)


@dataclass
class Params:
    type: int = C_SVC
    C: float = 1.0
    eps: float = 0.1
    gamma: float = 0.0
    tol: float = 1e-3
    max_iter: int = 0
    threads: int = 0
    kernel: int = RBF
    degree: int = 3
    coef0: float = 0.0

    def c(self, d: int) -> _Params:
        g = self.gamma if self.gamma > 0 else 1.0 / d
        return _Params(self.type, self.C, self.eps, g, self.tol,
                       self.max_iter, self.threads, self.kernel, self.degree,
                       self.coef0)


def _kparams(gamma: float, kind: int, degree: int, coef0: float) -> _Params:
    return _Params(C_SVC, 1.0, 0.0, gamma, 1.0, 0, 0, kind, degree, coef0)


@dataclass
class Result:
    alpha: np.ndarray
    F: np.ndarray
    iters: int
    gap: float
    m: float
    M: float
    b: float
    obj: float
    n_sv: int
    n_free: int
    status: int


def _res(alpha, F, r: _Result) -> Result:
    return Result(alpha, F, r.iters, r.gap, r.m, r.M, r.b, r.obj, r.n_sv,
                  r.n_free, r.status)


def num_vars(type_: int, n: int) -> int:
    return 2 * n if type_ == EPS_SVR else n


def kernel(A, B, gamma: float, kind: int = RBF, degree: int = 3,
           coef0: float = 0.0) -> np.ndarray:
    """Full kernel matrix K(a_i, b_j), fp64, by the direct definition."""
    A, B = _as_mat(A), _as_mat(B)
    out = np.empty((A.n, B.n), dtype=np.float64)
    kp = _kparams(gamma, kind, degree, coef0)
    rc = _load().orc_kernel(ct.byref(A.s), ct.byref(B.s), ct.byref(kp),
                            _ptr(out))
    assert rc == 0
    return out


def kernel_rows(X, gamma: float, idx, threads: int = 0, kind: int = RBF,
                degree: int = 3, coef0: float = 0.0) -> np.ndarray:
    """Kernel rows K(x_idx[j], X) -> (len(idx), n) fp64."""
    X = _as_mat(X)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty((len(idx), X.n), dtype=np.float64)
    kp = _kparams(gamma, kind, degree, coef0)
    rc = _load().orc_kernel_rows(ct.byref(X.s), ct.byref(kp), _ptr(idx),
                                 len(idx), threads, _ptr(out))
    assert rc == 0
    return out


def train(X, y, p: Params) -> Result:
    """Maximal-violating-pair SMO from alpha = 0 to gap <= tol."""
    X = _as_mat(X)
    y = np.ascontiguousarray(y, dtype=np.float32)
    N = num_vars(p.type, X.n)
    alpha = np.zeros(N, dtype=np.float64)
    F = np.zeros(X.n, dtype=np.float64)
    r = _Result()
    rc = _load().orc_train(ct.byref(X.s), _ptr(y), ct.byref(p.c(X.d)),
                           _ptr(alpha), _ptr(F), ct.byref(r))
    assert rc >= 0, rc
    return _res(alpha, F, r)


def solve(X, y, p: Params, alpha, F, max_steps: int = 0) -> Result:
    """Continue SMO from a given state for at most max_steps steps."""
    X = _as_mat(X)
    y = np.ascontiguousarray(y, dtype=np.float32)
    alpha = np.array(alpha, dtype=np.float64, copy=True)
    F = np.array(F, dtype=np.float64, copy=True)
    r = _Result()
    rc = _load().orc_solve(ct.byref(X.s), _ptr(y), ct.byref(p.c(X.d)),
                           max_steps, _ptr(alpha), _ptr(F), ct.byref(r))
    assert rc >= 0, rc
    return _res(alpha, F, r)


def state_summary(y, p: Params, alpha, F, d: int) -> Result:
    y = np.ascontiguousarray(y, dtype=np.float32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    F = np.ascontiguousarray(F, dtype=np.float64)
    r = _Result()
    _load().orc_state_summary(len(y), _ptr(y), ct.byref(p.c(d)), _ptr(alpha),
                              _ptr(F), ct.byref(r))
    return _res(alpha, F, r)


def responses(X, y, p: Params, alpha) -> np.ndarray:
    X = _as_mat(X)
    y = np.ascontiguousarray(y, dtype=np.float32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    F = np.empty(X.n, dtype=np.float64)
    rc = _load().orc_responses(ct.byref(X.s), _ptr(y), ct.byref(p.c(X.d)),
                               _ptr(alpha), _ptr(F))
    assert rc == 0
    return F


def select(y, p: Params, alpha, F, q: int, d: int = 1):
    """Working set of at most q variables -> (B, m, M)."""
    y = np.ascontiguousarray(y, dtype=np.float32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    F = np.ascontiguousarray(F, dtype=np.float64)
    B = np.empty(q, dtype=np.int32)
    nB = ct.c_int32()
    m = ct.c_double()
    M = ct.c_double()
    rc = _load().orc_select(len(y), _ptr(y), ct.byref(p.c(d)), _ptr(alpha),
                            _ptr(F), q, _ptr(B), ct.byref(nB), ct.byref(m),
                            ct.byref(M))
    assert rc == 0
    return B[: nB.value].copy(), m.value, M.value


def sample_of(type_: int, n: int, t):
    t = np.asarray(t)
    return np.where((type_ == EPS_SVR) & (t >= n), t - n, t)


def subproblem(X, y, p: Params, alpha, F, B, inner_tol: float,
               max_inner: int, KBB=None):
    """Inner maximal-violating-pair solve on the working set B.

    KBB defaults to the fp64 kernel block over the samples of B.
    Returns (alpha_B_new, steps)."""
    X = _as_mat(X)
    y = np.ascontiguousarray(y, dtype=np.float32)
    B = np.ascontiguousarray(B, dtype=np.int32)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    F = np.ascontiguousarray(F, dtype=np.float64)
    if KBB is None:
        sB = sample_of(p.type, X.n, B)
        XB = X.rows(sB)
        KBB = kernel(XB, XB, p.c(X.d).gamma, p.kernel, p.degree, p.coef0)
    KBB = np.ascontiguousarray(KBB, dtype=np.float64)
    out = np.empty(len(B), dtype=np.float64)
    steps = ct.c_int32()
    rc = _load().orc_subproblem(X.n, _ptr(y), ct.byref(p.c(X.d)), len(B),
                                _ptr(B), _ptr(alpha), _ptr(F), _ptr(KBB),
                                inner_tol, max_inner, _ptr(out),
                                ct.byref(steps))
    assert rc == 0
    return out, steps.value


def coefficients(type_: int, n: int, y, alpha) -> np.ndarray:
    """Per-sample expansion coefficient c_i (C-SVC: y_i a_i; SVR: a+ - a-)."""
    alpha = np.asarray(alpha, dtype=np.float64)
    if type_ == EPS_SVR:
        return alpha[:n] - alpha[n:]
    return np.where(np.asarray(y) > 0, 1.0, -1.0) * alpha


def decision(SV, coef, b: float, Xt, gamma: float, threads: int = 0,
             kind: int = RBF, degree: int = 3, coef0: float = 0.0):
    """D(x) = sum_i coef_i K(sv_i, x) + b, fp64 direct sums."""
    SV, Xt = _as_mat(SV), _as_mat(Xt)
    coef = np.ascontiguousarray(coef, dtype=np.float64)
    out = np.empty(Xt.n, dtype=np.float64)
    kp = _kparams(gamma, kind, degree, coef0)
    rc = _load().orc_decision(ct.byref(SV.s), _ptr(coef), b, ct.byref(Xt.s),
                              ct.byref(kp), threads, _ptr(out))
    assert rc == 0
    return out


def model_decision(X, y, p: Params, res: Result, Xt, threads: int = 0):
    """Decision values of a trained oracle state on test points."""
    X = _as_mat(X)
    c = coefficients(p.type, X.n, y, res.alpha)
    sv = np.nonzero(c)[0]
    if len(sv) == 0:
        return np.full(_as_mat(Xt).n, res.b)
    return decision(X.rows(sv), c[sv], res.b, Xt, p.c(X.d).gamma, threads,
                    p.kernel, p.degree, p.coef0)


def train_ovr(X, labels, n_classes: int, p: Params):
    """One-vs-rest multi-class: one binary C-SVC per class."""
    labels = np.asarray(labels)
    out = []
    for c in range(n_classes):
        yc = np.where(labels == c, 1.0, -1.0).astype(np.float32)
        out.append(train(X, yc, p))
    return out


# ---------------------------------------------------------------------------
# Scaling, k-fold cross-validation and metrics (Section 3's feature list:
# "scaling training data", "K-fold cross validation", "accuracy or
# correlation, mean square error"), by their definitions in fp64.
# ---------------------------------------------------------------------------

def scale_stats(X):
    """Per-column mean and sample standard deviation (n - 1 divisor), fp64.
    A constant column has sd 0 (it is left as it is)."""
    A = np.asarray(X, dtype=np.float64)
    mu = A.mean(axis=0)
    sd = np.sqrt(((A - mu) ** 2).sum(axis=0) / (A.shape[0] - 1))
    return mu, sd


def scale_apply(X, mu, sd):
    """(x - mu) / sd per column in fp64, rounded once to fp32; columns with
    sd 0 unchanged."""
    A = np.asarray(X, dtype=np.float64)
    s = np.where(sd > 0, sd, 1.0)
    m = np.where(sd > 0, mu, 0.0)
    return ((A - m) / s).astype(np.float32)


def train_scaled(X, y, p: Params, Xt):
    """Training on standardised features (and, for eps-SVR, targets) and the
    decision values of Xt in the units of the targets: (result, D)."""
    mu, sd = scale_stats(X)
    Xs, Xts = scale_apply(X, mu, sd), scale_apply(Xt, mu, sd)
    ys, y_mu, y_sd = np.asarray(y, np.float32), 0.0, 0.0
    if p.type == EPS_SVR:
        (y_mu,), (y_sd,) = scale_stats(np.asarray(y)[:, None])
        if y_sd > 0:
            ys = scale_apply(np.asarray(y)[:, None], np.array([y_mu]),
                             np.array([y_sd]))[:, 0]
    r = train(Xs, ys, p)
    D = model_decision(Xs, ys, p, r, Xts)
    if p.type == EPS_SVR and y_sd > 0:
        D = D * y_sd + y_mu
    return r, D


def _rows(X, idx):
    return X[idx] if not hasattr(X, "indptr") else X[idx]


def cross_validate(X, y, p: Params, k: int, fold=None, labels=None,
                   n_classes: int = 0):
    """Decision values of every row from the model trained on the rows of
    the other folds (fold[i] in [0, k); None: i mod k).  labels with
    n_classes: one-vs-rest, D is n x n_classes."""
    n = X.shape[0]
    fold = np.arange(n) % k if fold is None else np.asarray(fold)
    n_out = n_classes if labels is not None else 1
    D = np.zeros((n, n_out))
    for f in range(k):
        tr, te = np.nonzero(fold != f)[0], np.nonzero(fold == f)[0]
        Xtr, Xte = _rows(X, tr), _rows(X, te)
        for c in range(n_out):
            if labels is not None:
                yc = np.where(np.asarray(labels)[tr] == c, 1.0,
                              -1.0).astype(np.float32)
            else:
                yc = np.asarray(y, np.float32)[tr]
            r = train(Xtr, yc, p)
            D[te, c] = model_decision(Xtr, yc, p, r, Xte)
    return D[:, 0] if n_out == 1 else D


def metrics(type_: int, D, y=None, labels=None):
    """accuracy (C-SVC: D >= 0 is +1; one-vs-rest: argmax, ties to the
    lowest class), mse and squared correlation (eps-SVR), and the error
    that tuning minimises (1 - accuracy, or mse)."""
    D = np.asarray(D, dtype=np.float64)
    if labels is not None:
        acc = float(np.mean(np.argmax(D, axis=1) == np.asarray(labels)))
        return {"accuracy": acc, "error": 1.0 - acc}
    t = np.asarray(y, dtype=np.float64)
    if type_ == C_SVC:
        acc = float(np.mean(np.where(D >= 0, 1.0, -1.0) == t))
        return {"accuracy": acc, "error": 1.0 - acc}
    mse = float(np.mean((D - t) ** 2))
    n = len(t)
    num = n * (D @ t) - D.sum() * t.sum()
    den = (n * (D @ D) - D.sum() ** 2) * (n * (t @ t) - t.sum() ** 2)
    scc = float(num * num / den) if den > 0 else 0.0
    return {"mse": mse, "scc": scc, "error": mse}
