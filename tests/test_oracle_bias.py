"""Pins for the bias rule of the oracle (the paper does not define b; the
rule below is LIBSVM's).

b is the mean of the keys v_t over the free variables (0 < a_t < C); when
no variable is free, the midpoint (m + M) / 2 of the largest I_up key and
the smallest I_low key.  The states below are constructed by hand so that
the two rules give different numbers: each expected value is worked out in
the comments from the definitions v_t = r_t - F_smp(t), r_t = y_t (C-SVC)
or z_i -/+ eps (eps-SVR copy (i,+) / (i,-)), I_up = {y=+1, a<C} u {y=-1,
a>0}, I_low = {y=+1, a>0} u {y=-1, a<C}.
"""
import numpy as np
import pytest

import oracle
from oracle import C_SVC, EPS_SVR, Params

# C-SVC, C = 1:  y = + - + - + -,  F below, so v = y - F =
#   [0.8, -0.9, 0.5, -1.4, 1.7, -1.05]
Y6 = np.array([1, -1, 1, -1, 1, -1], dtype=np.float32)
F6 = np.array([0.2, -0.1, 0.5, 0.4, -0.7, 0.05])


def test_bias_is_mean_over_free_keys_svc():
    # alpha = [0.3, 0.3, 1, 0, 0, 1] (y^T a = 0): free t0, t1 ->
    # b = (0.8 - 0.9) / 2 = -0.05.  I_up = {t0, t4 (y=+1, a<1), t1, t5
    # (y=-1, a>0)} -> m = 1.7; I_low = {t0, t2 (y=+1, a>0), t1, t3 (y=-1,
    # a<1)} -> M = -1.4; the midpoint would be 0.15.
    a = np.array([0.3, 0.3, 1.0, 0.0, 0.0, 1.0])
    p = Params(C_SVC, C=1.0, gamma=1.0, tol=1e-3)
    r = oracle.state_summary(Y6, p, a, F6, d=1)
    assert r.n_free == 2
    assert r.m == pytest.approx(1.7, abs=1e-15)
    assert r.M == pytest.approx(-1.4, abs=1e-15)
    assert r.b == pytest.approx(-0.05, abs=1e-15)


def test_bias_is_midpoint_without_free_svc():
    # alpha = [1, 1, 0, 0, 0, 0]: no free variable.  I_up = {t2, t4 (y=+1,
    # a<1), t1 (y=-1, a>0)} -> m = 1.7; I_low = {t0 (y=+1, a>0), t3, t5
    # (y=-1, a<1)} -> M = -1.4; b = (1.7 - 1.4) / 2 = 0.15.
    a = np.array([1.0, 1.0, 0.0, 0.0, 0.0, 0.0])
    p = Params(C_SVC, C=1.0, gamma=1.0, tol=1e-3)
    r = oracle.state_summary(Y6, p, a, F6, d=1)
    assert r.n_free == 0
    assert r.b == pytest.approx(0.15, abs=1e-15)


def test_bias_is_mean_over_free_keys_svr():
    # eps-SVR, eps = 0.1, C = 1, z = [1, 0, -0.5, 2], F = [0.6, 0.3, -0.2,
    # 0.4].  Copies (i,+) = t0..t3: v = z - eps - F = [0.3, -0.4, -0.4,
    # 1.5]; copies (i,-) = t4..t7: v = z + eps - F = [0.5, -0.2, -0.2, 1.7].
    # alpha: t0 = 0.4, t6 = 0.4, the rest 0 (sum a+ = sum a-).  Free: t0,
    # t6 -> b = (0.3 - 0.2) / 2 = 0.05.  I_up = {t0..t3 (y=+1, a<C), t6
    # (y=-1, a>0)} -> m = 1.5; I_low = {t0 (y=+1, a>0), t4..t7 (y=-1, a<C)}
    # -> M = -0.2; the midpoint would be 0.65.
    z = np.array([1.0, 0.0, -0.5, 2.0], dtype=np.float32)
    F = np.array([0.6, 0.3, -0.2, 0.4])
    a = np.zeros(8)
    a[0] = a[6] = 0.4
    p = Params(EPS_SVR, C=1.0, eps=0.1, gamma=1.0, tol=1e-3)
    r = oracle.state_summary(z, p, a, F, d=1)
    assert r.n_free == 2
    assert r.m == pytest.approx(1.5, abs=1e-7)
    assert r.M == pytest.approx(-0.2, abs=1e-7)
    assert r.b == pytest.approx(0.05, abs=1e-7)


def test_bias_is_midpoint_without_free_svr():
    # Same targets and responses, alpha: t1 = 1 = C and t5 = 1 (copies of
    # sample 1 at the bound), the rest 0.  I_up = {t0, t2, t3 (y=+1, a<C),
    # t5 (y=-1, a>0)} -> m = 1.5; I_low = {t1 (y=+1, a>0), t4, t6, t7 (y=-1,
    # a<C)} -> M = -0.4 (t1); b = (1.5 - 0.4) / 2 = 0.55.
    z = np.array([1.0, 0.0, -0.5, 2.0], dtype=np.float32)
    F = np.array([0.6, 0.3, -0.2, 0.4])
    a = np.zeros(8)
    a[1] = a[5] = 1.0
    p = Params(EPS_SVR, C=1.0, eps=0.1, gamma=1.0, tol=1e-3)
    r = oracle.state_summary(z, p, a, F, d=1)
    assert r.n_free == 0
    assert r.m == pytest.approx(1.5, abs=1e-7)
    assert r.M == pytest.approx(-0.4, abs=1e-7)
    assert r.b == pytest.approx(0.55, abs=1e-7)
