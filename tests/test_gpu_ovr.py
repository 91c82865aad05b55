"""One-vs-rest multi-class (C4 recipe, d = 784) on the GPU against the
oracle: per-class dual objective (1e-4 relative), decision values (1e-3
absolute) and argmax labels (>= 99.9 % equal)."""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, Params
from paper_1706_05544_amd import native as nv
from paper_1706_05544_amd import workloads

pytestmark = pytest.mark.gpu


def test_c4_recipe_ovr_small():
    w = workloads.c4(n=3000, n_test=600)
    p = Params(C_SVC, C=w.C, gamma=w.gamma, tol=w.tol)
    refs = oracle.train_ovr(w.X, w.y, w.n_classes, p)
    m = nv.svm_train_ovr(w.X, w.y, w.n_classes, C=w.C, gamma=w.gamma,
                         tol=w.tol)
    assert m.n_outputs == 10
    D = nv.svm_predict(m, w.Xt)
    assert D.shape == (600, 10)
    Dref = np.empty_like(D)
    for c, r in enumerate(refs):
        info = m.info(c)
        assert info["status"] == nv.SVM_OK
        assert info["dual_obj"] == pytest.approx(r.obj, rel=1e-4)
        yc = np.where(w.y == c, 1.0, -1.0).astype(np.float32)
        Dref[:, c] = oracle.model_decision(w.X, yc, p, r, w.Xt)
        idx, coef, alpha = nv.svm_model_get(m, c, with_alpha=True)
        cc = oracle.coefficients(C_SVC, w.n, yc, alpha)
        assert list(idx) == list(np.nonzero(cc)[0])
    assert np.max(np.abs(D - Dref)) <= 1e-3
    L = nv.svm_predict_labels(m, w.Xt)
    Lref = np.argmax(Dref, axis=1)
    assert np.mean(L == Lref) >= 0.999
    assert np.mean(L == w.yt) > 0.9


def test_ovr_labels_on_device():
    import torch
    w = workloads.c4(n=800, n_test=100)
    mh = nv.svm_train_ovr(w.X, w.y, 10, C=w.C, gamma=w.gamma)
    md = nv.svm_train_ovr(torch.from_numpy(w.X).cuda(),
                          torch.from_numpy(w.y).cuda(), 10, C=w.C,
                          gamma=w.gamma)
    Lh = nv.svm_predict_labels(mh, w.Xt)
    Ld = nv.svm_predict_labels(md, torch.from_numpy(w.Xt).cuda()).cpu().numpy()
    assert np.array_equal(Lh, Ld)
