"""Python binding of libmi355svm.so: argument marshalling only.

Every entry point of ``include/mi355svm.h`` has a function of the same name
here.  Host inputs are NumPy arrays; device inputs are torch tensors on a
ROCm device (PyTorch is used for device memory and streams only).  All
computation happens in the library's HIP kernels; if the library is not
built, loading fails loudly instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as ct
import os
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmi355svm.so")

SVM_OK = 0
SVM_W_MAX_ITER = 1
SVM_W_NOT_CONVERGED = 2
SVM_E_INVALID = -1
SVM_E_UNSUPPORTED = -2
SVM_E_NOMEM = -3
SVM_E_DEVICE = -4
SVM_E_INTERNAL = -5

SVM_C_SVC = 0
SVM_EPS_SVR = 1
SVM_KERNEL_LINEAR, SVM_KERNEL_POLY, SVM_KERNEL_RBF, SVM_KERNEL_SIGMOID = range(4)
SVM_DENSE = 0
SVM_CSR = 1

# every symbol the header declares
EXPORTS = [
    "svm_params_default", "svm_train", "svm_train_ovr", "svm_predict",
    "svm_predict_labels", "svm_model_get_info", "svm_model_get",
    "svm_model_free", "svm_last_error", "svm_cross_validate", "svm_tune",
    "svm_test_solver_create",
    "svm_test_solver_free", "svm_test_set_state", "svm_test_get_state",
    "svm_test_select", "svm_test_rows", "svm_test_subproblem",
    "svm_test_apply", "svm_test_iterate", "svm_test_finish",
    "svm_predict_noalloc", "svm_cache_release",
]


class SvmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("status %d: %s" % (status, msg))
        self.status = status


class svm_matrix(ct.Structure):
    _fields_ = [("layout", ct.c_int32), ("on_device", ct.c_int32),
                ("n", ct.c_int64), ("d", ct.c_int64),
                ("values", ct.c_void_p), ("ld", ct.c_int64),
                ("row_ptr", ct.c_void_p), ("col_idx", ct.c_void_p),
                ("nnz", ct.c_int64)]


class svm_params(ct.Structure):
    _fields_ = [("type", ct.c_int32), ("kernel", ct.c_int32),
                ("C", ct.c_double), ("epsilon", ct.c_double),
                ("gamma", ct.c_double), ("tol", ct.c_double),
                ("max_iter", ct.c_int64), ("working_set", ct.c_int32),
                ("device", ct.c_int32), ("cache_bytes", ct.c_int64),
                ("stream", ct.c_void_p), ("check_every", ct.c_int32),
                ("inner_ratio", ct.c_double), ("max_inner", ct.c_int32),
                ("profile", ct.c_int32), ("coef0", ct.c_double),
                ("degree", ct.c_int32), ("scale", ct.c_int32),
                ("alpha0", ct.c_void_p), ("lockstep", ct.c_int32),
                ("fused", ct.c_int32)]


class svm_cv_stats(ct.Structure):
    _fields_ = [("folds", ct.c_int32), ("status", ct.c_int32),
                ("n", ct.c_int64), ("iters", ct.c_int64),
                ("accuracy", ct.c_double), ("mse", ct.c_double),
                ("scc", ct.c_double), ("error", ct.c_double),
                ("kernel_rows", ct.c_int64), ("row_kernel_ms", ct.c_double),
                ("row_kernel_launches", ct.c_int64),
                ("row_kernel_bytes", ct.c_double)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


class svm_model_info(ct.Structure):
    _fields_ = [("type", ct.c_int32), ("n_outputs", ct.c_int32),
                ("n_train", ct.c_int64), ("n_features", ct.c_int64),
                ("n_sv", ct.c_int64), ("gamma", ct.c_double),
                ("kernel", ct.c_int32), ("degree", ct.c_int32),
                ("coef0", ct.c_double),
                ("status", ct.c_int32), ("n_sv_output", ct.c_int64),
                ("n_bounded", ct.c_int64), ("iters", ct.c_int64),
                ("gap", ct.c_double), ("b", ct.c_double),
                ("dual_obj", ct.c_double), ("kernel_rows", ct.c_int64),
                ("cache_hits", ct.c_int64), ("cache_fills", ct.c_int64),
                ("train_ms", ct.c_double),
                ("row_kernel_ms", ct.c_double),
                ("row_kernel_launches", ct.c_int64),
                ("row_kernel_rows", ct.c_int64),
                ("row_kernel_bytes", ct.c_double),
                ("cached_kernel_ms", ct.c_double),
                ("cached_kernel_launches", ct.c_int64),
                ("cached_kernel_bytes", ct.c_double),
                ("select_kernel_ms", ct.c_double),
                ("select_kernel_launches", ct.c_int64)]

    def as_dict(self) -> dict:
        return {k: getattr(self, k) for k, _ in self._fields_}


_lib = None


def load(path: Optional[str] = None):
    """Load the built library; raise if it is missing (no fallback path)."""
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(
            "libmi355svm.so is not built; run __graft_entry__.build() or "
            "python -m paper_1706_05544_amd.build")
    try:
        # torch bundles its own copy of the HIP runtime under the same soname;
        # loading torch first makes the library bind to that copy, so that
        # one runtime serves both and device pointers are shared.
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ct.CDLL(path)
    P = ct.POINTER
    vp = ct.c_void_p
    lib.svm_params_default.argtypes = [P(svm_params)]
    lib.svm_params_default.restype = None
    lib.svm_train.argtypes = [P(svm_matrix), vp, P(svm_params), P(vp)]
    lib.svm_train_ovr.argtypes = [P(svm_matrix), vp, ct.c_int32,
                                  P(svm_params), P(vp)]
    lib.svm_predict.argtypes = [vp, P(svm_matrix), vp]
    lib.svm_predict_labels.argtypes = [vp, P(svm_matrix), vp]
    lib.svm_model_get_info.argtypes = [vp, ct.c_int32, P(svm_model_info)]
    lib.svm_model_get.argtypes = [vp, ct.c_int32, vp, vp, vp]
    lib.svm_model_free.argtypes = [vp]
    lib.svm_model_free.restype = None
    lib.svm_cache_release.argtypes = [ct.c_int32, P(ct.c_int64)]
    lib.svm_cross_validate.argtypes = [P(svm_matrix), vp, vp, ct.c_int32,
                                       P(svm_params), ct.c_int32, vp, vp,
                                       P(svm_cv_stats)]
    lib.svm_tune.argtypes = [P(svm_matrix), vp, vp, ct.c_int32,
                             P(svm_params), ct.c_int32, vp, ct.c_int32, vp, vp,
                             vp, vp, P(ct.c_int32)]
    lib.svm_last_error.restype = ct.c_char_p
    lib.svm_last_error.argtypes = []
    lib.svm_test_solver_create.argtypes = [P(svm_matrix), vp, P(svm_params),
                                           P(vp)]
    lib.svm_test_solver_free.argtypes = [vp]
    lib.svm_test_solver_free.restype = None
    lib.svm_test_set_state.argtypes = [vp, vp, vp]
    lib.svm_test_get_state.argtypes = [vp, vp, vp]
    lib.svm_test_select.argtypes = [vp, vp, P(ct.c_int32), P(ct.c_double),
                                    P(ct.c_double)]
    lib.svm_test_rows.argtypes = [vp, vp, ct.c_int32, vp]
    lib.svm_test_subproblem.argtypes = [vp, vp, ct.c_int32, ct.c_double,
                                        ct.c_int32, vp, P(ct.c_int32)]
    lib.svm_test_apply.argtypes = [vp, vp, ct.c_int32, vp]
    lib.svm_test_iterate.argtypes = [vp, ct.c_int64, P(ct.c_int64),
                                     P(ct.c_double)]
    lib.svm_predict_noalloc.argtypes = [vp, P(svm_matrix), vp, vp]
    lib.svm_test_finish.argtypes = [vp, ct.c_int32, P(ct.c_double),
                                    P(ct.c_double), P(ct.c_double),
                                    P(ct.c_int32)]
    for name in EXPORTS:  # fail now, not at first use, if one is missing
        getattr(lib, name)
    _lib = lib
    return lib


def svm_last_error() -> str:
    return load().svm_last_error().decode()


def _check(rc: int) -> int:
    if rc < 0:
        raise SvmError(rc, svm_last_error())
    return rc


def _is_torch(x) -> bool:
    return type(x).__module__.startswith("torch")


def _torch_sparse_csr():
    import torch
    return torch.sparse_csr


def _np_ptr(a: np.ndarray) -> int:
    return a.ctypes.data


class _Mat:
    """svm_matrix for a NumPy array (host), a scipy CSR matrix (host) or a
    contiguous torch tensor on the GPU (device); keeps its buffers alive."""

    def __init__(self, X):
        self.keep = []
        m = svm_matrix()
        if _is_torch(X) and X.layout == _torch_sparse_csr():
            import torch
            assert X.is_cuda and X.dim() == 2
            rp = X.crow_indices().to(torch.int64).contiguous()
            ci = X.col_indices().to(torch.int32).contiguous()
            cv = X.values().to(torch.float32).contiguous()
            self.keep += [rp, ci, cv]
            m.layout, m.on_device = SVM_CSR, 1
            m.n, m.d = X.shape
            m.values, m.row_ptr, m.col_idx = (cv.data_ptr(), rp.data_ptr(),
                                              ci.data_ptr())
            m.nnz = cv.numel()
            self.device = True
        elif _is_torch(X):
            import torch
            assert X.is_cuda and X.dtype == torch.float32 and X.dim() == 2
            X = X.contiguous()
            self.keep.append(X)
            m.layout, m.on_device = SVM_DENSE, 1
            m.n, m.d = X.shape
            m.values, m.ld = X.data_ptr(), X.shape[1]
            self.device = True
        elif hasattr(X, "indptr"):
            data = np.ascontiguousarray(X.data, dtype=np.float32)
            ip = np.ascontiguousarray(X.indptr, dtype=np.int64)
            ix = np.ascontiguousarray(X.indices, dtype=np.int32)
            self.keep += [data, ip, ix]
            m.layout, m.on_device = SVM_CSR, 0
            m.n, m.d = X.shape
            m.values, m.row_ptr, m.col_idx = _np_ptr(data), _np_ptr(ip), _np_ptr(ix)
            m.nnz = len(data)
            self.device = False
        else:
            A = np.ascontiguousarray(X, dtype=np.float32)
            assert A.ndim == 2
            self.keep.append(A)
            m.layout, m.on_device = SVM_DENSE, 0
            m.n, m.d = A.shape
            m.values, m.ld = (_np_ptr(A) if A.size else None), A.shape[1]
            self.device = False
        self.s = m


def _vec(v, dtype, device: bool):
    if device:
        import torch
        tdt = {np.float32: torch.float32, np.int32: torch.int32}[dtype]
        t = v if _is_torch(v) else torch.as_tensor(np.asarray(v))
        t = t.to(device="cuda", dtype=tdt).contiguous()
        return t, t.data_ptr()
    a = np.ascontiguousarray(v, dtype=dtype)
    return a, _np_ptr(a)


def svm_params_default(**overrides) -> svm_params:
    p = svm_params()
    load().svm_params_default(ct.byref(p))
    for k, v in overrides.items():
        if not hasattr(p, k):
            raise TypeError("unknown svm_params field %r" % k)
        setattr(p, k, v)
    return p


class Model:
    """Owns an svm_model*; freed with svm_model_free."""

    def __init__(self, ptr: int, status: int):
        self.ptr = ptr
        self.status = status

    def __del__(self):
        if getattr(self, "ptr", None) and _lib is not None:
            _lib.svm_model_free(self.ptr)
            self.ptr = None

    def info(self, output: int = 0) -> dict:
        return svm_model_get_info(self, output)

    @property
    def n_outputs(self) -> int:
        return self.info(0)["n_outputs"]


def _stream_of(device: bool):
    if not device:
        return None
    import torch
    return torch.cuda.current_stream().cuda_stream


def svm_train(X, y, params: Optional[svm_params] = None, alpha0=None,
              **kw) -> Model:
    p = params or svm_params_default(**kw)
    a0 = None
    if alpha0 is not None:  # warm start (host values, kept alive here)
        a0 = np.ascontiguousarray(alpha0, dtype=np.float64)
        p.alpha0 = _np_ptr(a0)
    M = _Mat(X)
    if M.device and not kw.get("stream") and not (params and params.stream):
        p.stream = _stream_of(True)
    yv, yp = _vec(y, np.float32, M.device)
    out = ct.c_void_p()
    rc = _check(load().svm_train(ct.byref(M.s), yp, ct.byref(p),
                                 ct.byref(out)))
    return Model(out.value, rc)


def svm_train_ovr(X, labels, n_classes: int,
                  params: Optional[svm_params] = None, **kw) -> Model:
    p = params or svm_params_default(**kw)
    M = _Mat(X)
    if M.device and not kw.get("stream") and not (params and params.stream):
        p.stream = _stream_of(True)
    lv, lp = _vec(labels, np.int32, M.device)
    out = ct.c_void_p()
    rc = _check(load().svm_train_ovr(ct.byref(M.s), lp, n_classes,
                                     ct.byref(p), ct.byref(out)))
    return Model(out.value, rc)


def svm_predict(model: Model, X):
    M = _Mat(X)
    n_out = model.n_outputs
    m = M.s.n
    if M.device:
        import torch
        D = torch.empty((m, n_out), dtype=torch.float64, device="cuda")
        ptr = D.data_ptr() if m else None
    else:
        D = np.empty((m, n_out), dtype=np.float64)
        ptr = _np_ptr(D) if m else None
    _check(load().svm_predict(model.ptr, ct.byref(M.s), ptr))
    return D[:, 0] if n_out == 1 else D


def svm_predict_noalloc(model: Model, X, out=None, stream=None):
    """svm_predict_noalloc: X a dense torch tensor on the GPU; the decision
    values go to `out` (a float64 tensor of m x n_outputs, allocated here
    when None) on `stream` (torch's current stream when None), not waited
    for.  Returns out."""
    import torch
    M = _Mat(X)
    if not M.device:
        raise SvmError(SVM_E_UNSUPPORTED, "svm_predict_noalloc takes a "
                       "tensor in device memory")
    n_out = model.n_outputs
    m = M.s.n
    if out is None:
        out = torch.empty((m, n_out), dtype=torch.float64, device=X.device)
    assert out.dtype == torch.float64 and out.is_contiguous()
    assert out.numel() == m * n_out
    st = stream if stream is not None else torch.cuda.current_stream()
    _check(load().svm_predict_noalloc(model.ptr, ct.byref(M.s),
                                      out.data_ptr() if m else None,
                                      st.cuda_stream))
    return out


def svm_predict_labels(model: Model, X):
    M = _Mat(X)
    m = M.s.n
    if M.device:
        import torch
        L = torch.empty((m,), dtype=torch.int32, device="cuda")
        ptr = L.data_ptr() if m else None
    else:
        L = np.empty((m,), dtype=np.int32)
        ptr = _np_ptr(L) if m else None
    _check(load().svm_predict_labels(model.ptr, ct.byref(M.s), ptr))
    return L


def svm_cache_release(device: int = -1) -> int:
    """Frees the row-cache memory the library keeps between trainings on
    `device` (-1: every device); returns the bytes freed."""
    freed = ct.c_int64(0)
    _check(load().svm_cache_release(device, ct.byref(freed)))
    return freed.value


def svm_model_get_info(model: Model, output: int = 0) -> dict:
    info = svm_model_info()
    _check(load().svm_model_get_info(model.ptr, output, ct.byref(info)))
    return info.as_dict()


def _cv_inputs(X, y, labels, fold):
    # X host or device; labels, targets and folds on the host
    M = _Mat(X)
    if hasattr(y, "cpu"):
        y = y.cpu().numpy()
    if hasattr(labels, "cpu"):
        labels = labels.cpu().numpy()
    yv = None if y is None else np.ascontiguousarray(y, dtype=np.float32)
    lv = None if labels is None else np.ascontiguousarray(labels,
                                                          dtype=np.int32)
    fv = None if fold is None else np.ascontiguousarray(fold, dtype=np.int32)
    return (M, yv, lv, fv,
            None if yv is None else _np_ptr(yv),
            None if lv is None else _np_ptr(lv),
            None if fv is None else _np_ptr(fv))


def svm_cross_validate(X, y=None, labels=None, n_classes: int = 0,
                       k: int = 10, fold=None,
                       params: Optional[svm_params] = None, **kw):
    """k-fold cross-validation -> (decision values n x n_outputs, stats)."""
    p = params or svm_params_default(**kw)
    M, yv, lv, fv, yp, lp, fp = _cv_inputs(X, y, labels, fold)
    if M.device and not kw.get("stream") and not (params and params.stream):
        p.stream = _stream_of(True)
    n_out = n_classes if labels is not None else 1
    D = np.empty((M.s.n, n_out), dtype=np.float64)
    st = svm_cv_stats()
    rc = _check(load().svm_cross_validate(ct.byref(M.s), yp, lp, n_classes,
                                          ct.byref(p), k, fp, _np_ptr(D),
                                          ct.byref(st)))
    out = st.as_dict()
    out["rc"] = rc
    return (D[:, 0] if n_out == 1 else D), out


def svm_tune(X, y=None, labels=None, n_classes: int = 0, k: int = 10,
             fold=None, C=None, gamma=None, epsilon=None,
             params: Optional[svm_params] = None, **kw):
    """Grid tuning by k-fold cross-validation -> (errors, best index)."""
    p = params or svm_params_default(**kw)
    M, yv, lv, fv, yp, lp, fp = _cv_inputs(X, y, labels, fold)
    if M.device and not kw.get("stream") and not (params and params.stream):
        p.stream = _stream_of(True)
    arrs = [None if a is None else np.ascontiguousarray(a, dtype=np.float64)
            for a in (C, gamma, epsilon)]
    n_grid = max(len(a) for a in arrs if a is not None)
    err = np.empty(n_grid, dtype=np.float64)
    best = ct.c_int32()
    _check(load().svm_tune(ct.byref(M.s), yp, lp, n_classes, ct.byref(p), k,
                           fp, n_grid,
                           *[None if a is None else _np_ptr(a) for a in arrs],
                           _np_ptr(err), ct.byref(best)))
    return err, best.value


def svm_model_get(model: Model, output: int = 0, with_alpha: bool = False):
    """-> (sv_idx int32, coef fp64, alpha fp64 or None)."""
    info = svm_model_get_info(model, output)
    k = info["n_sv_output"]
    idx = np.empty(max(k, 1), dtype=np.int32)
    coef = np.empty(max(k, 1), dtype=np.float64)
    alpha = None
    if with_alpha:
        N = info["n_train"] * (2 if info["type"] == SVM_EPS_SVR else 1)
        alpha = np.empty(N, dtype=np.float64)
    _check(load().svm_model_get(model.ptr, output, _np_ptr(idx),
                                _np_ptr(coef),
                                _np_ptr(alpha) if alpha is not None else None))
    return idx[:k], coef[:k], alpha


class Solver:
    """The svm_test_* hooks: a solver whose state can be set and stepped."""

    def __init__(self, X, y, params: Optional[svm_params] = None, **kw):
        p = params or svm_params_default(**kw)
        M = _Mat(X)
        yv, yp = _vec(y, np.float32, False)
        out = ct.c_void_p()
        _check(load().svm_test_solver_create(ct.byref(M.s), yp, ct.byref(p),
                                             ct.byref(out)))
        self.ptr = out.value
        self.n = M.s.n
        self.N = self.n * (2 if p.type == SVM_EPS_SVR else 1)

    def __del__(self):
        if getattr(self, "ptr", None) and _lib is not None:
            _lib.svm_test_solver_free(self.ptr)
            self.ptr = None

    def set_state(self, alpha, F):
        a = np.ascontiguousarray(alpha, dtype=np.float64)
        f = np.ascontiguousarray(F, dtype=np.float64)
        _check(load().svm_test_set_state(self.ptr, _np_ptr(a), _np_ptr(f)))

    def get_state(self):
        a = np.empty(self.N, dtype=np.float64)
        f = np.empty(self.n, dtype=np.float64)
        _check(load().svm_test_get_state(self.ptr, _np_ptr(a), _np_ptr(f)))
        return a, f

    def select(self):
        B = np.empty(64, dtype=np.int32)
        nB = ct.c_int32()
        m = ct.c_double()
        M = ct.c_double()
        _check(load().svm_test_select(self.ptr, _np_ptr(B), ct.byref(nB),
                                      ct.byref(m), ct.byref(M)))
        return B[: nB.value].copy(), m.value, M.value

    def rows(self, samples):
        s = np.ascontiguousarray(samples, dtype=np.int32)
        out = np.empty((len(s), self.n), dtype=np.float32)
        _check(load().svm_test_rows(self.ptr, _np_ptr(s), len(s),
                                    _np_ptr(out)))
        return out

    def subproblem(self, B, inner_tol: float, max_inner: int):
        b = np.ascontiguousarray(B, dtype=np.int32)
        out = np.empty(len(b), dtype=np.float64)
        steps = ct.c_int32()
        _check(load().svm_test_subproblem(self.ptr, _np_ptr(b), len(b),
                                          inner_tol, max_inner, _np_ptr(out),
                                          ct.byref(steps)))
        return out, steps.value

    def apply(self, B, alpha_B):
        b = np.ascontiguousarray(B, dtype=np.int32)
        a = np.ascontiguousarray(alpha_B, dtype=np.float64)
        _check(load().svm_test_apply(self.ptr, _np_ptr(b), len(b), _np_ptr(a)))

    def iterate(self, k: int):
        it = ct.c_int64()
        gap = ct.c_double()
        _check(load().svm_test_iterate(self.ptr, k, ct.byref(it),
                                       ct.byref(gap)))
        return it.value, gap.value

    def finish(self, max_passes: int = 3):
        """End a training on the current state: (gap, b, obj, status)."""
        gap, b, obj = ct.c_double(), ct.c_double(), ct.c_double()
        st = ct.c_int32()
        _check(load().svm_test_finish(self.ptr, max_passes, ct.byref(gap),
                                      ct.byref(b), ct.byref(obj),
                                      ct.byref(st)))
        return gap.value, b.value, obj.value, st.value
