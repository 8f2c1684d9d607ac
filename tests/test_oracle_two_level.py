"""Pins of the oracle's two-level controller (xfer, then location; NO-OP
ends the episode) against forced choices, the masks and the softmax
distributions the Gumbel-max draws must follow."""

import numpy as np
from scipy import stats

from oracle import wm

N, L = 3, 5


def _logits(n, seed):
    return np.random.default_rng(seed).normal(size=(n, N + 1 + L))


def test_forced_choice_and_flat_index():
    n = 40
    xm = np.zeros((n, N + 1), np.uint8)
    xm[:, 2] = 1
    lm = np.zeros((n, N, L), np.uint8)
    lm[:, 2, 4] = 1
    lm[:, 0, :] = 1  # other xfers' locations do not matter
    a, _, _ = wm.two_level_action(_logits(n, 1), xm, lm, seed=3, traj=np.arange(n), step=0, N=N, L=L)
    np.testing.assert_array_equal(a, np.full(n, 2 * L + 4))


def test_noop_and_empty_cases():
    n = 20
    lg = _logits(n, 2)
    xm = np.zeros((n, N + 1), np.uint8)
    xm[:, N] = 1  # only the NO-OP
    lm = np.ones((n, N, L), np.uint8)
    a, _, _ = wm.two_level_action(lg, xm, lm, seed=1, traj=np.arange(n), step=0, N=N, L=L)
    assert np.all(a == -2)
    a, _, _ = wm.two_level_action(lg, np.zeros_like(xm), lm, seed=1, traj=np.arange(n), step=0, N=N, L=L)
    assert np.all(a == -1)
    xm[:, N] = 0
    xm[:, 1] = 1
    lm[:, 1, :] = 0  # the only xfer has no valid location
    a, _, _ = wm.two_level_action(lg, xm, lm, seed=1, traj=np.arange(n), step=0, N=N, L=L)
    assert np.all(a == -1)


def test_locations_valid_under_the_chosen_xfer():
    n = 500
    rng = np.random.default_rng(5)
    xm = (rng.random((n, N + 1)) < 0.6).astype(np.uint8)
    xm[:, 0] = 1
    lm = (rng.random((n, N, L)) < 0.5).astype(np.uint8)
    lm[:, :, 0] = 1
    a, _, _ = wm.two_level_action(_logits(n, 6), xm, lm, seed=7, traj=np.arange(n), step=4, N=N, L=L)
    pos = a >= 0
    x, l = a[pos] // L, a[pos] % L
    assert np.all(xm[pos, x] == 1) and np.all(lm[np.nonzero(pos)[0], x, l] == 1)
    assert np.all(xm[a == -2, N] == 1)


def test_pick_frequencies_follow_the_masked_softmaxes():
    n = 40000
    one = np.array([0.3, -0.5, 1.1, 0.2, 0.4, -1.0, 0.9, 0.0, 0.5])  # N+1 xfer then L location logits
    lg = np.tile(one, (n, 1))
    xm = np.array([1, 0, 1, 1], np.uint8)[None].repeat(n, 0)
    lm = np.ones((n, N, L), np.uint8)
    lm[:, 2, 1] = 0
    a, _, _ = wm.two_level_action(lg, xm, lm, seed=11, traj=np.arange(n), step=2, N=N, L=L)
    x = np.where(a == -2, N, a // L)
    px = wm.masked_softmax(one[:N + 1], xm[0])
    cnt = np.bincount(x, minlength=N + 1)
    assert stats.chisquare(cnt[px > 0], n * px[px > 0]).pvalue > 1e-4
    assert cnt[1] == 0
    sel = x == 2  # locations of xfer 2 follow the softmax over its valid locations
    pl = wm.masked_softmax(one[N + 1:], lm[0, 2])
    cl = np.bincount(a[sel] % L, minlength=L)
    assert stats.chisquare(cl[pl > 0], sel.sum() * pl[pl > 0]).pvalue > 1e-4
    assert cl[1] == 0


def test_rollout_noop_ends_the_trajectory():
    Z, H, K, B, T = 4, 6, 2, 6, 4
    A = N * L
    rng = np.random.default_rng(9)
    w = dict(W_g=rng.normal(size=(4 * H, Z + A + H)) * 0.3, b_g=np.zeros(4 * H),
             W_m=rng.normal(size=(3 * Z * K, H)) * 0.3, b_m=np.zeros(3 * Z * K),
             w_r=rng.normal(size=H), b_r=np.zeros(1), w_d=rng.normal(size=H), b_d=np.array([-9.0]),
             W_c=rng.normal(size=(N + 1 + L, Z + H)), b_c=np.zeros(N + 1 + L))
    xm = np.ones((B, N + 1), np.uint8)
    xm[0, :N] = 0  # row 0 can only stop
    lm = np.ones((B, N, L), np.uint8)
    r = wm.rollout(w, dict(Z=Z, H=H, A=A, K=K), rng.normal(size=(B, Z)), (xm, lm), T=T, seed=2,
                   two_level=(N, L))
    assert r["actions"][0, 0] == -2 and r["rewards"][0, 0] == 0 and r["dones"][0, 0] == 1
    assert np.all(r["actions"][1:, 0] == -1)
    np.testing.assert_array_equal(r["z_out"][1:, 0], np.broadcast_to(r["z_out"][0, 0], (T, Z)))
    live = r["actions"] >= 0
    assert live[:, 1:].any() and np.all(r["actions"][live] < A)


def test_controller_step_factored_probabilities():
    """The two-level controller step's probabilities: the xfer softmax over
    the valid xfers, then the location softmax over the locations valid for
    the picked xfer (zero after a NO-OP or no pick); the action's parts carry
    positive probability; against a direct float64 softmax of the logits."""
    from paper_2205_01435_amd import workloads as wl
    Z, H, K, n = 8, 16, 2, 300
    rng = np.random.default_rng(9)
    w = wl.make_weights(rng, Z, H, N * L, K, 10)
    a_ = np.sqrt(6.0 / (Z + H + N + 1 + L))
    w["W_c"] = rng.uniform(-a_, a_, size=(N + 1 + L, Z + H))
    w["b_c"] = rng.normal(size=N + 1 + L)
    dims = dict(Z=Z, H=H, A=N * L, K=K)
    z = rng.normal(size=(n, Z))
    h = np.tanh(rng.normal(size=(n, H)))
    xm = (rng.random((n, N + 1)) < 0.6).astype(np.uint8)
    xm[:5] = 0
    xm[5:10] = 0
    xm[5:10, N] = 1  # NO-OP only
    lm = (rng.random((n, N, L)) < 0.5).astype(np.uint8)
    r = wm.controller_step(w, dims, z, h, (xm, lm), seed=4, step=2, two_level=(N, L))
    p = r["probs"]
    assert p.shape == (n, N + 1 + L)
    logits = np.concatenate([z, h], axis=1) @ np.asarray(w["W_c"]).T + w["b_c"]
    for b in range(n):
        px = p[b, :N + 1]
        if xm[b].any():
            e = np.where(xm[b] != 0, np.exp(logits[b, :N + 1] - logits[b, :N + 1][xm[b] != 0].max()), 0)
            np.testing.assert_allclose(px, e / e.sum(), rtol=1e-12, atol=1e-15)
        else:
            assert np.all(px == 0)
        x = r["xfer"][b]
        pl = p[b, N + 1:]
        if 0 <= x < N and lm[b, x].any():
            e = np.where(lm[b, x] != 0, np.exp(logits[b, N + 1:] - logits[b, N + 1:][lm[b, x] != 0].max()), 0)
            np.testing.assert_allclose(pl, e / e.sum(), rtol=1e-12, atol=1e-15)
        else:
            assert np.all(pl == 0)
        a = r["action"][b]
        if a >= 0:
            assert px[a // L] > 0 and pl[a % L] > 0 and xm[b, a // L] and lm[b, a // L, a % L]
        elif a == -2:
            assert x == N
    assert np.all(r["action"][:5] == -1) and np.all(r["action"][5:10] == -2)
