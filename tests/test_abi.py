"""C ABI: the library loads here (no GPU), exports every declared symbol,
its ctypes mirror matches the C layout, and argument validation reports
errors before any device call; with valid arguments and no GPU it returns
SVM_E_DEVICE cleanly."""
import os
import re
import subprocess

import ctypes as ct

import numpy as np
import pytest

from paper_1706_05544_amd import native as nv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mi355svm.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(svm_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = nv.load()
    names = _declared()
    assert len(names) >= 15
    assert set(names) == set(nv.EXPORTS)
    out = subprocess.run(["nm", "-D", "--defined-only", nv.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r" T (svm_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(lib, n)


def test_struct_layout_matches_header(tmp_path):
    prog = tmp_path / "layout.c"
    prog.write_text(r'''
#include <stdio.h>
#include <stddef.h>
#include "mi355svm.h"
int main(void) {
  printf("%zu %zu %zu\n", sizeof(svm_matrix), sizeof(svm_params),
         sizeof(svm_model_info));
  printf("%zu %zu %zu %zu %zu %zu %zu %zu %zu %zu %zu\n",
         offsetof(svm_params, stream),
         offsetof(svm_params, profile), offsetof(svm_model_info, train_ms),
         offsetof(svm_matrix, nnz), offsetof(svm_params, coef0),
         offsetof(svm_params, degree), offsetof(svm_model_info, coef0),
         offsetof(svm_params, scale), sizeof(svm_cv_stats),
         offsetof(svm_cv_stats, error), offsetof(svm_params, lockstep));
  return 0;
}
''')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER),
                    str(prog), "-o", str(exe)], check=True)
    a, b = subprocess.run([str(exe)], capture_output=True, text=True,
                          check=True).stdout.split("\n")[:2]
    import ctypes as ct
    assert [int(x) for x in a.split()] == [
        ct.sizeof(nv.svm_matrix), ct.sizeof(nv.svm_params),
        ct.sizeof(nv.svm_model_info)]
    assert [int(x) for x in b.split()] == [
        nv.svm_params.stream.offset, nv.svm_params.profile.offset,
        nv.svm_model_info.train_ms.offset, nv.svm_matrix.nnz.offset,
        nv.svm_params.coef0.offset, nv.svm_params.degree.offset,
        nv.svm_model_info.coef0.offset, nv.svm_params.scale.offset,
        ct.sizeof(nv.svm_cv_stats), nv.svm_cv_stats.error.offset,
        nv.svm_params.lockstep.offset]


def test_params_default():
    p = nv.svm_params_default()
    assert p.type == nv.SVM_C_SVC and p.kernel == nv.SVM_KERNEL_RBF
    assert p.C == 1.0 and p.epsilon == 0.1 and p.gamma == 0.0
    assert p.tol == 1e-3 and p.working_set == 16 and p.device == 0
    assert p.coef0 == 0.0 and p.degree == 3


def _x(n=8, d=3):
    return np.random.default_rng(0).standard_normal((n, d)).astype(np.float32)


def _y(n=8):
    return np.where(np.arange(n) % 2 == 0, 1.0, -1.0).astype(np.float32)


@pytest.mark.parametrize("kw,code", [
    (dict(C=0.0), nv.SVM_E_INVALID),
    (dict(C=float("nan")), nv.SVM_E_INVALID),
    (dict(tol=0.0), nv.SVM_E_INVALID),
    (dict(gamma=-1.0), nv.SVM_E_INVALID),
    (dict(epsilon=-0.1), nv.SVM_E_INVALID),
    (dict(working_set=3), nv.SVM_E_INVALID),
    (dict(working_set=66), nv.SVM_E_INVALID),
    (dict(working_set=0), nv.SVM_E_INVALID),
    (dict(type=7), nv.SVM_E_INVALID),
    (dict(kernel=9), nv.SVM_E_INVALID),
    (dict(kernel=-1), nv.SVM_E_INVALID),
    (dict(kernel=nv.SVM_KERNEL_POLY, degree=0), nv.SVM_E_INVALID),
    (dict(kernel=nv.SVM_KERNEL_POLY, degree=65), nv.SVM_E_INVALID),
    (dict(kernel=nv.SVM_KERNEL_SIGMOID, coef0=float("inf")),
     nv.SVM_E_INVALID),
    (dict(inner_ratio=1.5), nv.SVM_E_INVALID),
    (dict(scale=2), nv.SVM_E_INVALID),
])
def test_invalid_params(kw, code):
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(), _y(), **kw)
    assert e.value.status == code
    assert nv.svm_last_error()


def test_invalid_labels_and_shapes():
    y = _y()
    y[3] = 0.5
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(), y)
    assert e.value.status == nv.SVM_E_INVALID and "+1 or -1" in str(e.value)
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(), np.ones(8, np.float32))
    assert "both classes" in str(e.value)
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(1, 3), np.ones(1, np.float32))
    assert e.value.status == nv.SVM_E_INVALID
    z = _y()
    z[0] = np.inf
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(), z, type=nv.SVM_EPS_SVR)
    assert "finite" in str(e.value)
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train_ovr(_x(), np.array([0, 1, 2, 0, 1, 2, 0, 5]), 3)
    assert e.value.status == nv.SVM_E_INVALID
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train_ovr(_x(), np.zeros(8, np.int32), 3)
    assert "every class" in str(e.value)


def test_null_arguments_are_rejected():
    lib = nv.load()
    import ctypes as ct
    out = ct.c_void_p()
    p = nv.svm_params_default()
    assert lib.svm_train(None, None, ct.byref(p), ct.byref(out)) == \
        nv.SVM_E_INVALID
    M = nv._Mat(_x())
    assert lib.svm_train(ct.byref(M.s), None, ct.byref(p), ct.byref(out)) \
        == nv.SVM_E_INVALID
    assert lib.svm_predict(None, ct.byref(M.s), None) == nv.SVM_E_INVALID
    assert lib.svm_model_get_info(None, 0, None) == nv.SVM_E_INVALID
    lib.svm_model_free(None)


def test_csr_arguments_are_checked_before_the_device():
    # pointer and count checks of a CSR matrix happen on the host (its
    # structure, sortedness and finiteness are checked on the device)
    import scipy.sparse as sp
    lib = nv.load()
    y = np.ascontiguousarray(_y(), dtype=np.float32)
    p = nv.svm_params_default()
    out = ct.c_void_p()
    for field, value in (("row_ptr", None), ("nnz", -1), ("col_idx", None),
                         ("values", None)):
        M = nv._Mat(sp.csr_matrix(_x()))
        setattr(M.s, field, value)
        st = lib.svm_train(ct.byref(M.s), y.ctypes.data, ct.byref(p),
                           ct.byref(out))
        assert st == nv.SVM_E_INVALID, (field, st)


@pytest.mark.skipif(os.path.exists("/dev/kfd"), reason="a GPU is present")
def test_no_device_is_a_clean_error():
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(), _y())
    assert e.value.status == nv.SVM_E_DEVICE
    assert "device" in nv.svm_last_error()


@pytest.mark.parametrize("kw,code", [
    (dict(k=1), nv.SVM_E_INVALID),
    (dict(k=9), nv.SVM_E_INVALID),                      # more folds than rows
    (dict(k=2, fold=[0, 1, 2, 0, 1, 0, 1, 0]), nv.SVM_E_INVALID),
    (dict(k=3, fold=[0, 1, 0, 1, 0, 1, 0, 1]), nv.SVM_E_INVALID),  # empty fold
    (dict(k=2, scale=3), nv.SVM_E_INVALID),
    (dict(k=2, lockstep=5), nv.SVM_E_INVALID),
    (dict(k=2, lockstep=-1), nv.SVM_E_INVALID),
    (dict(k=2, lockstep=2, working_set=32), nv.SVM_E_UNSUPPORTED),
])
def test_cross_validate_invalid(kw, code):
    with pytest.raises(nv.SvmError) as e:
        nv.svm_cross_validate(_x(), _y(), **kw)
    assert e.value.status == code


def test_cross_validate_needs_exactly_one_truth():
    with pytest.raises(nv.SvmError) as e:
        nv.svm_cross_validate(_x(), _y(), labels=np.zeros(8, np.int32),
                              n_classes=2, k=2)
    assert e.value.status == nv.SVM_E_INVALID
    with pytest.raises(nv.SvmError) as e:
        nv.svm_tune(_x(), _y(), k=2, C=[1.0, -1.0])  # C <= 0 in the grid
    assert e.value.status == nv.SVM_E_INVALID


@pytest.mark.parametrize("a0", [
    [-0.1, 0.1, 0, 0, 0, 0, 0, 0],        # below 0
    [2.0, 2.0, 0, 0, 0, 0, 0, 0],         # above C = 1
    [0.5, 0.0, 0, 0, 0, 0, 0, 0],         # y^T a != 0 (labels +1, -1, ...)
    [float("nan"), 0, 0, 0, 0, 0, 0, 0],
])
def test_warm_start_invalid(a0):
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train(_x(), _y(), alpha0=np.array(a0, np.float64))
    assert e.value.status == nv.SVM_E_INVALID
    assert "alpha0" in str(e.value)


def test_lockstep_needs_dense_features():
    # checked before the device: the same error with or without a GPU
    import scipy.sparse as sp
    X = sp.csr_matrix(_x())
    with pytest.raises(nv.SvmError) as e:
        nv.svm_cross_validate(X, _y(), k=2, lockstep=2)
    assert e.value.status == nv.SVM_E_UNSUPPORTED
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train_ovr(X, np.arange(8, dtype=np.int32) % 2, 2, lockstep=3)
    assert e.value.status == nv.SVM_E_UNSUPPORTED
    with pytest.raises(nv.SvmError) as e:
        nv.svm_train_ovr(_x(), np.arange(8, dtype=np.int32) % 2, 2,
                         lockstep=9)
    assert e.value.status == nv.SVM_E_INVALID
