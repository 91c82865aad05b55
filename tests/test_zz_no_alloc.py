"""svm_predict_noalloc (no device allocation, staging in a static per-device
array) against svm_predict: the same kernels, so the decision values must
be the same bits.  Two calls in a row on the same GPU array, the second
with fewer rows, for each model kind: rows used in place (d a multiple of
4), rows copied with zero padding (d = 7), a model trained on scaled
features (and eps-SVR targets), and a one-vs-rest model with 784 features
whose query rows take several chunks of the array."""
import numpy as np
import pytest
import torch

from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def _model(kind):
    if kind == "inplace":
        w = workloads.c1(n=1500, n_test=10)
        m = nv.svm_train(w.X, w.y, C=w.C, gamma=w.gamma, tol=w.tol)
        return m, w.d
    if kind == "padded":
        w = workloads.c1(n=1500, n_test=10)
        X = np.ascontiguousarray(w.X[:, :7])
        m = nv.svm_train(X, w.y, C=w.C, gamma=1.0 / 7, tol=w.tol)
        return m, 7
    if kind == "scaled_svr":
        w = workloads.c2(n=1200, n_test=10)
        m = nv.svm_train(w.X, w.y, type=nv.SVM_EPS_SVR, C=w.C, epsilon=w.eps,
                         gamma=w.gamma, tol=w.tol, scale=1)
        return m, w.d
    if kind == "ovr_chunks":
        w = workloads.make("C4", n=2000, n_test=10)
        m = nv.svm_train_ovr(w.X, w.y, w.n_classes, C=w.C, gamma=w.gamma,
                             tol=w.tol)
        return m, w.d
    raise ValueError(kind)


@pytest.mark.parametrize("kind,m1,m2", [("inplace", 3000, 700),
                                        ("padded", 2500, 1),
                                        ("scaled_svr", 2000, 333),
                                        ("ovr_chunks", 25000, 9000)])
def test_noalloc_matches_predict(kind, m1, m2):
    model, d = _model(kind)
    rng = np.random.default_rng(m1 + m2)
    for m in (m1, m2):
        Xt = torch.from_numpy(rng.random((m, d), dtype=np.float32)
                              * 2.0 - 0.5).to("cuda:0")
        ref = nv.svm_predict(model, Xt)
        if ref.ndim == 1:
            ref = ref[:, None]
        out = torch.full((m, model.n_outputs), float("nan"),
                         dtype=torch.float64, device="cuda:0")
        nv.svm_predict_noalloc(model, Xt, out)
        torch.cuda.synchronize()
        assert torch.equal(out, ref), (kind, m,
                                       float((out - ref).abs().max()))


def test_noalloc_rejects_host_and_csr_rows():
    w = workloads.c1(n=300, n_test=10)
    model = nv.svm_train(w.X, w.y, C=w.C, gamma=w.gamma, tol=w.tol)
    with pytest.raises(nv.SvmError) as e:
        nv.svm_predict_noalloc(model, w.Xt)
    assert e.value.status == nv.SVM_E_UNSUPPORTED
    Xd = torch.from_numpy(np.ascontiguousarray(w.Xt[:, :5])).to("cuda:0")
    with pytest.raises(nv.SvmError) as e:
        nv.svm_predict_noalloc(model, Xd)
    assert e.value.status == nv.SVM_E_INVALID
