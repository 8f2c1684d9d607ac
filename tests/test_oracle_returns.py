"""Pins of the return-scan oracle against closed forms and explicit sums.

Each pin is computed by a formula other than the oracle's recursion: a
geometric series, a direct double sum over future steps with the
continuation product written out, the one-step TD error, or the identity
between GAE(1) and the bootstrapped discounted return.
"""

import numpy as np
import pytest

from oracle import returns as oret


def _direct_returns(r, d, gamma, bootstrap=None):
    """G_t = sum_{i >= t} gamma^(i-t) r_i prod_{t <= u < i} (1 - d_u)
    (+ gamma^(T-t) prod_{t <= u < T} (1 - d_u) V_T), as an explicit sum."""
    T, B = r.shape
    G = np.zeros((T, B))
    for t in range(T):
        for b in range(B):
            s, live = 0.0, 1.0
            for i in range(t, T):
                s += gamma ** (i - t) * live * r[i, b]
                live *= 1.0 - d[i, b]
            if bootstrap is not None:
                s += gamma ** (T - t) * live * bootstrap[b]
            G[t, b] = s
    return G


def _data(seed, T=9, B=5, pdone=0.2):
    rng = np.random.default_rng(seed)
    r = rng.normal(size=(T, B))
    d = (rng.random((T, B)) < pdone).astype(np.uint8)
    V = rng.normal(size=(T + 1, B))
    return r, d, V


def test_geometric_series():
    T, gamma, c = 12, 0.9, 0.7
    r = np.full((T, 3), c)
    G, A = oret.returns(r, np.zeros((T, 3), np.uint8), gamma)
    t = np.arange(T)[:, None]
    np.testing.assert_allclose(G, c * (1 - gamma ** (T - t)) / (1 - gamma) * np.ones((1, 3)), rtol=1e-13)
    assert A is None


def test_gamma_zero_is_the_reward():
    r, d, _ = _data(1)
    G, _ = oret.returns(r, d, 0.0)
    np.testing.assert_array_equal(G, r)


@pytest.mark.parametrize("seed,gamma", [(2, 0.99), (3, 0.5), (4, 1.0)])
def test_direct_sum_with_dones(seed, gamma):
    r, d, _ = _data(seed)
    G, _ = oret.returns(r, d, gamma)
    np.testing.assert_allclose(G, _direct_returns(r, d, gamma), rtol=1e-12, atol=1e-12)


def test_done_cuts_the_tail():
    # a done at step 3: steps 0..3 see rewards 0..3 only, whatever follows
    T = 8
    r = np.arange(1.0, T + 1)[:, None]
    d = np.zeros((T, 1), np.uint8)
    d[3] = 1
    G, _ = oret.returns(r, d, 0.5)
    assert G[3, 0] == 4.0
    assert G[0, 0] == 1 + 0.5 * 2 + 0.25 * 3 + 0.125 * 4
    G2, _ = oret.returns(np.concatenate([r[:4], np.full((T - 4, 1), 99.0)]), d, 0.5)
    np.testing.assert_array_equal(G[:4], G2[:4])


@pytest.mark.parametrize("seed,gamma", [(5, 0.97), (6, 0.8)])
def test_gae_lambda_one_is_the_bootstrapped_return(seed, gamma):
    r, d, V = _data(seed)
    ret, A = oret.returns(r, d, gamma, values=V, lam=1.0)
    np.testing.assert_allclose(ret, _direct_returns(r, d, gamma, bootstrap=V[-1]), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(A, ret - V[:-1], rtol=1e-12, atol=1e-12)


def test_gae_lambda_zero_is_the_td_error():
    r, d, V = _data(7)
    gamma = 0.9
    _, A = oret.returns(r, d, gamma, values=V, lam=0.0)
    np.testing.assert_allclose(A, r + gamma * (1.0 - d) * V[1:] - V[:-1], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("seed,gamma,lam", [(8, 0.99, 0.95), (9, 0.7, 0.3)])
def test_gae_direct_sum(seed, gamma, lam):
    # A_t = sum_l (gamma lam)^l delta_{t+l} prod_{t <= u < t+l} (1 - d_u)
    r, d, V = _data(seed)
    _, A = oret.returns(r, d, gamma, values=V, lam=lam)
    delta = r + gamma * (1.0 - d) * V[1:] - V[:-1]
    np.testing.assert_allclose(A, _direct_returns(delta, d, gamma * lam), rtol=1e-12, atol=1e-12)
