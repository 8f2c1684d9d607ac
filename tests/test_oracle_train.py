"""Pins of the training-step oracle: the hand-written gradient against
central finite differences of the forward oracle's loss (a different code
path), a closed form of the mixture gradient, the learning-rate schedule's
values and Adam's first steps in closed form."""

import numpy as np
import pytest

from oracle import train as otr
from oracle import wm

DIMS = dict(Z=4, H=5, A=3, K=2)


def _case(seed=0, T=3, B=2, Z=4, H=5, A=3, K=2, lengths=None):
    rng = np.random.default_rng(seed)
    w = dict(W_g=rng.normal(size=(4 * H, Z + A + H)) * 0.6, b_g=rng.normal(size=4 * H) * 0.3,
             W_m=rng.normal(size=(3 * Z * K, H)) * 0.6, b_m=rng.normal(size=3 * Z * K) * 0.3,
             w_r=rng.normal(size=H), b_r=rng.normal(size=1), w_d=rng.normal(size=H),
             b_d=rng.normal(size=1), W_c=np.zeros((A, Z + H)), b_c=np.zeros(A))
    z = rng.normal(size=(T + 1, B, Z))
    a = rng.integers(0, A, size=(T, B))
    a[0, 0] = -1  # a step without an action
    r = rng.normal(size=(T, B))
    d = (rng.random((T, B)) < 0.4).astype(np.uint8)
    return w, dict(Z=Z, H=H, A=A, K=K), z, a, r, d, lengths


@pytest.mark.parametrize("seed,lengths", [(1, None), (2, np.array([3, 1])), (3, np.array([2, 0]))])
def test_gradient_matches_finite_differences(seed, lengths):
    w, dims, z, a, r, d, ln = _case(seed, lengths=lengths)
    L, g = otr.loss_and_grads(w, dims, z, a, r, d, ln)
    assert abs(L - otr.loss(w, dims, z, a, r, d, ln)) < 1e-12
    eps = 1e-6
    for k in otr.PARAMS:
        base = np.asarray(w[k], np.float64)
        num = np.zeros(base.size)
        for i in range(base.size):
            wp = dict(w)
            wm_ = dict(w)
            xp = base.copy().reshape(-1)
            xm = base.copy().reshape(-1)
            xp[i] += eps
            xm[i] -= eps
            wp[k] = xp.reshape(base.shape)
            wm_[k] = xm.reshape(base.shape)
            num[i] = (otr.loss(wp, dims, z, a, r, d, ln) - otr.loss(wm_, dims, z, a, r, d, ln)) / (2 * eps)
        np.testing.assert_allclose(np.asarray(g[k]).reshape(-1), num, rtol=2e-5, atol=1e-8, err_msg=k)


def test_single_gaussian_mean_gradient_closed_form():
    """K = 1, one step: d L / d b_mu_j = -(x_j - mu_j) / (sigma_j^2 N Z)."""
    w, dims, z, a, r, d, _ = _case(4, T=1, B=3, K=1)
    _, g = otr.loss_and_grads(w, dims, z, a, r, d)
    f = wm.nll(w, dims, z, a, r, d)
    Z, K, H = dims["Z"], dims["K"], dims["H"]
    hn = f["h_trace"][0]                                # [B, H]
    m = hn @ np.asarray(w["W_m"]).T + w["b_m"]          # [B, 3Z]
    mu, ls = m[:, Z:2 * Z], m[:, 2 * Z:]
    want = (-(z[1] - mu) / np.exp(2 * ls)).sum(axis=0) / (3 * Z)
    np.testing.assert_allclose(g["b_m"][Z:2 * Z], want, rtol=1e-12)


def test_polynomial_learning_rate():
    assert otr.poly_lr(0, 1e-3, 1e-5) == 1e-3
    assert otr.poly_lr(5000, 1e-3, 1e-5) == 1e-5
    assert abs(otr.poly_lr(2500, 1e-3, 1e-5) - ((1e-3 - 1e-5) / 4 + 1e-5)) < 1e-18
    assert otr.poly_lr(9000, 1e-3, 1e-5) == 1e-5


def test_adam_first_steps_closed_form():
    p = {"x": np.array([1.0, -2.0, 0.5])}
    g = {"x": np.array([0.3, -0.01, 2.0])}
    st = {}
    p1 = otr.adam_step(p, g, st, lr=0.1)
    # bias-corrected moments are g and g^2: a step of lr g / (|g| + eps)
    np.testing.assert_allclose(p1["x"], p["x"] - 0.1 * g["x"] / (np.abs(g["x"]) + 1e-8), rtol=1e-12)
    p2 = otr.adam_step(p1, g, st, lr=0.1)  # a constant gradient keeps the step
    np.testing.assert_allclose(p2["x"], p1["x"] - 0.1 * g["x"] / (np.abs(g["x"]) + 1e-8), rtol=1e-9)
    assert st["t"] == 2
