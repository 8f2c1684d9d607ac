"""Pins of the oracle against closed forms, library routines and invariants.

Each test fixes a part of ``oracle.wm`` with something other than the oracle
itself, chosen so that a plausible slip (a dropped term, a wrong sign, a
transposed operand, a wrong gate block or layout index) fails one of them.
"""

import math

import numpy as np
import pytest
import torch
from scipy import special, stats

from oracle import bf16 as obf
from oracle import philox as ph
from oracle import wm
from paper_2205_01435_amd import workloads as wl

DIMS = dict(Z=4, H=6, A=5, K=3)


def _weights(seed=0, Z=4, H=6, A=5, K=3, T=10, scale=1.0):
    rng = np.random.default_rng(seed)
    w = wl.make_weights(rng, Z, H, A, K, T)
    for k in ("W_g", "W_m", "W_c", "w_r", "w_d"):
        w[k] = (w[k] * scale).astype(np.float32)
    w["b_g"] = rng.normal(size=4 * H).astype(np.float32) * 0.3
    w["b_m"] = rng.normal(size=3 * Z * K).astype(np.float32) * 0.3
    w["b_c"] = rng.normal(size=A).astype(np.float32) * 0.3
    w["b_r"] = np.float32(0.2)
    return w


# --------------------------------------------------------------------------
# bf16 storage rounding
# --------------------------------------------------------------------------

def test_bf16_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.normal(size=20000) * 10.0 ** rng.integers(-30, 30, size=20000),
        np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.4e38, 1e-40, -1e-42]),
    ]).astype(np.float32)
    # exact ties: low 16 bits == 0x8000, with both parities of bit 16
    tie_bits = (rng.integers(0, 2 ** 15, size=2000, dtype=np.uint32) << 17) | 0x8000
    tie_bits |= (rng.integers(0, 2, size=2000, dtype=np.uint32) << 16)
    tie_bits = (tie_bits & 0x7FFFFFFF) | (0x3F000000 & ~0)  # keep exponents moderate
    x = np.concatenate([x, tie_bits.view(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = obf.round_bf16(x)
    assert np.array_equal(got, ref, equal_nan=True)
    assert np.isnan(obf.round_bf16(np.array([np.nan], np.float32)))[0]


def test_q_identity_for_fp32():
    x = np.random.default_rng(1).normal(size=100)
    assert np.array_equal(obf.q(x, "fp32"), x)


# --------------------------------------------------------------------------
# controller (section 3.4) and masking (section 3.1.3)
# --------------------------------------------------------------------------

def test_controller_logits_match_torch_linear():
    w = _weights()
    wb = wm.weight_blocks(w, **DIMS, dtype="fp32")
    rng = np.random.default_rng(2)
    z, h = rng.normal(size=(7, 4)), rng.normal(size=(7, 6))
    ref = torch.nn.functional.linear(torch.from_numpy(np.concatenate([z, h], 1)),
                                     torch.from_numpy(w["W_c"].astype(np.float64)),
                                     torch.from_numpy(w["b_c"].astype(np.float64))).numpy()
    np.testing.assert_allclose(wm.controller_logits(wb, z, h, "fp32"), ref, rtol=1e-13, atol=1e-13)


def test_masked_softmax_vs_scipy_and_zero_on_masked():
    rng = np.random.default_rng(3)
    logits = rng.normal(size=(50, 9)) * 3
    mask = (rng.random((50, 9)) < 0.4).astype(np.uint8)
    mask[0] = 0
    mask[1] = 1
    p = wm.masked_softmax(logits, mask)
    assert np.all(p[mask == 0] == 0.0)
    assert np.all(p[0] == 0.0)
    for b in range(1, 50):
        v = mask[b] != 0
        if v.any():
            np.testing.assert_allclose(p[b, v], special.softmax(logits[b, v]), rtol=1e-13)
            assert abs(p[b].sum() - 1.0) < 1e-12


def test_gumbel_max_distribution_matches_masked_softmax():
    """Gumbel-max over Philox uniforms samples softmax over the valid set."""
    A = 6
    logits = np.array([0.3, -1.0, 2.0, 0.0, 1.1, -0.4])
    mask = np.array([1, 1, 0, 1, 1, 0], np.uint8)
    n = 200000
    u = ph.stream_uniforms(11, traj=np.arange(n), step=0, stream=0, n=A)
    a, margin, _ = wm.argmax_fp32(logits + wm.gumbel(u), mask != 0)
    counts = np.bincount(a, minlength=A)
    assert counts[2] == 0 and counts[5] == 0  # masked actions are never drawn
    p = special.softmax(logits[mask != 0])
    res = stats.chisquare(counts[mask != 0], p * n)
    assert res.pvalue > 1e-4
    assert np.all(margin >= 0)


def test_argmax_ties_and_empty():
    s = np.array([[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0], [1.0, 2.0, 3.0, 4.0]])
    v = np.array([[1, 1, 1, 1], [0, 1, 1, 1], [0, 0, 0, 0]], bool)
    idx, margin, _ = wm.argmax_fp32(s, v)
    assert idx.tolist() == [1, 1, -1]
    assert margin[0] == 0.0
    # decided on float32-rounded scores: a float64-only gap is a tie
    idx, margin, _ = wm.argmax_fp32(np.array([[1.0, 1.0 + 1e-12]]), True)
    assert idx[0] == 0 and 0 < margin[0] < 1e-11


# --------------------------------------------------------------------------
# LSTM core of the MDN-RNN (section 3.3.2)
# --------------------------------------------------------------------------

def test_lstm_step_matches_torch_lstmcell():
    Z, H, A = 4, 6, 5
    w = _weights()
    wb = wm.weight_blocks(w, Z, H, A, 3, "fp32")
    rng = np.random.default_rng(4)
    B = 9
    z, h, c = rng.normal(size=(B, Z)), rng.normal(size=(B, H)), rng.normal(size=(B, H))
    a = rng.integers(0, A, size=B)
    g = wm.gate_preactivations(wb, z, h, a, "fp32")
    h2, c2 = wm.lstm_cell(g, c)
    cell = torch.nn.LSTMCell(Z + A, H).double()
    W = w["W_g"].astype(np.float64)
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W[:, :Z + A]))
        cell.weight_hh.copy_(torch.from_numpy(W[:, Z + A:]))
        cell.bias_ih.copy_(torch.from_numpy(w["b_g"].astype(np.float64)))
        cell.bias_hh.zero_()
        x = torch.from_numpy(np.concatenate([z, np.eye(A)[a]], 1))
        rh, rc = cell(x, (torch.from_numpy(h), torch.from_numpy(c)))
    np.testing.assert_allclose(h2, rh.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(c2, rc.numpy(), rtol=1e-12, atol=1e-13)


def test_lstm_zero_weights_closed_form():
    rng = np.random.default_rng(5)
    c = rng.normal(size=(3, 8)) * 2
    h2, c2 = wm.lstm_cell(np.zeros((3, 32)), c)
    np.testing.assert_allclose(c2, 0.5 * c, rtol=1e-15)
    np.testing.assert_allclose(h2, 0.5 * np.tanh(0.5 * c), rtol=1e-15)


def test_no_action_contributes_zero_column():
    Z, H, A = 4, 6, 5
    w = _weights()
    wb = wm.weight_blocks(w, Z, H, A, 3, "fp32")
    rng = np.random.default_rng(6)
    z, h = rng.normal(size=(2, Z)), rng.normal(size=(2, H))
    g_none = wm.gate_preactivations(wb, z, h, np.array([-1, A]), "fp32")
    ref = z @ w["W_g"][:, :Z].T.astype(np.float64) + h @ w["W_g"][:, Z + A:].T + w["b_g"]
    np.testing.assert_allclose(g_none, ref, rtol=1e-13)


# --------------------------------------------------------------------------
# mixture head (section 3.3.2)
# --------------------------------------------------------------------------

def _nll_inputs(Z, H, A, K, T, B, seed=0):
    w = wl.Workload("t", "nll", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype="fp32", seed=seed)
    return wl.make_nll_inputs(w)


def test_nll_k1_is_gaussian_logpdf():
    """With one component log pi = 0 for any logit and the mixture
    log-likelihood is the Gaussian log-density (scipy.stats.norm)."""
    Z, H, A, K, T, B = 4, 6, 5, 1, 3, 4
    d = _nll_inputs(Z, H, A, K, T, B)
    w = d["weights"]
    w["b_m"] = np.random.default_rng(1).normal(size=3 * Z * K).astype(np.float32)
    out = wm.nll(w, dict(Z=Z, H=H, A=A, K=K), d["z"], d["actions"], d["rewards"], d["dones"])
    hf = out["h_trace"].reshape(T * B, H)
    m = hf @ w["W_m"].T.astype(np.float64) + w["b_m"]
    mu, ls = m[:, Z:2 * Z], m[:, 2 * Z:3 * Z]
    ref = stats.norm.logpdf(d["z"][1:].reshape(T * B, Z), loc=mu, scale=np.exp(ls)).sum(1)
    np.testing.assert_allclose(out["loglik"].ravel(), ref, rtol=1e-12)


def test_nll_mixture_vs_direct_sum_and_scipy_logsumexp():
    Z, H, A, K, T, B = 4, 6, 5, 3, 3, 5
    d = _nll_inputs(Z, H, A, K, T, B, seed=3)
    w = d["weights"]
    out = wm.nll(w, dict(Z=Z, H=H, A=A, K=K), d["z"], d["actions"], d["rewards"], d["dones"])
    hf = out["h_trace"].reshape(T * B, H)
    m = (hf @ w["W_m"].T.astype(np.float64) + w["b_m"]).reshape(T * B, 3, Z, K)
    pi = special.softmax(m[:, 0], axis=-1)
    x = d["z"][1:].reshape(T * B, Z)[..., None]
    dens = pi * stats.norm.pdf(x, loc=m[:, 1], scale=np.exp(m[:, 2]))
    np.testing.assert_allclose(out["loglik"].ravel(), np.log(dens.sum(-1)).sum(-1), rtol=1e-11)
    lse = special.logsumexp(np.log(pi) + stats.norm.logpdf(x, m[:, 1], np.exp(m[:, 2])), axis=-1)
    np.testing.assert_allclose(out["loglik"].ravel(), lse.sum(-1), rtol=1e-12)
    np.testing.assert_allclose(wm.logsumexp(m[:, 0], -1), special.logsumexp(m[:, 0], -1),
                               rtol=1e-14)


def test_reward_se_and_done_bce_vs_torch():
    Z, H, A, K, T, B = 4, 6, 5, 2, 4, 3
    d = _nll_inputs(Z, H, A, K, T, B, seed=4)
    w = d["weights"]
    w["b_d"] = np.float32(0.7)
    out = wm.nll(w, dict(Z=Z, H=H, A=A, K=K), d["z"], d["actions"], d["rewards"], d["dones"])
    hf = out["h_trace"]
    rho_r = hf @ w["w_r"].astype(np.float64) + float(w["b_r"])
    rho_d = hf @ w["w_d"].astype(np.float64) + float(w["b_d"])
    np.testing.assert_allclose(out["reward_se"], (rho_r - d["rewards"]) ** 2, rtol=1e-12)
    ref = torch.nn.functional.binary_cross_entropy_with_logits(
        torch.from_numpy(rho_d), torch.from_numpy(d["dones"].astype(np.float64)),
        reduction="none").numpy()
    np.testing.assert_allclose(out["done_bce"], ref, rtol=1e-12)


def test_nll_padding_and_means():
    Z, H, A, K, T, B = 4, 6, 5, 2, 5, 4
    d = _nll_inputs(Z, H, A, K, T, B, seed=5)
    dims = dict(Z=Z, H=H, A=A, K=K)
    full = wm.nll(d["weights"], dims, d["z"], d["actions"], d["rewards"], d["dones"])
    lengths = np.array([5, 0, 2, 3])
    pad = wm.nll(d["weights"], dims, d["z"], d["actions"], d["rewards"], d["dones"],
                 lengths=lengths)
    valid = np.arange(T)[:, None] < lengths[None, :]
    for k in ("loglik", "reward_se", "done_bce"):
        np.testing.assert_array_equal(pad[k][~valid], 0.0)
        np.testing.assert_allclose(pad[k][valid], full[k][valid], rtol=1e-14)
    N = lengths.sum()
    np.testing.assert_allclose(pad["means"], [-full["loglik"][valid].sum() / (N * Z),
                                              full["reward_se"][valid].sum() / N,
                                              full["done_bce"][valid].sum() / N], rtol=1e-13)


def test_mixture_weights_sum_to_one_and_temperature_limits():
    rng = np.random.default_rng(8)
    x = rng.normal(size=(100, 7)) * 4
    for tau in (0.25, 1.0, 1.5, 3.0):
        p = wm.mixture_weights(x, tau)
        assert np.all(np.abs(p.sum(-1) - 1.0) < 1e-12)
    np.testing.assert_allclose(wm.mixture_weights(x, 1.0), special.softmax(x, axis=-1), rtol=1e-13)
    np.testing.assert_allclose(wm.mixture_weights(x, 1e12), 1.0 / 7, rtol=1e-9)
    # tau -> 0 concentrates on the argmax
    p0 = wm.mixture_weights(x, 1e-6)
    assert np.array_equal(p0.argmax(-1), x.argmax(-1)) and np.all(p0.max(-1) > 1 - 1e-9)


def test_component_pick_frequencies_follow_temperature_softmax():
    """Gumbel-max on logit/tau samples Categorical(softmax(logit/tau))."""
    K, n = 4, 200000
    logits = np.array([0.5, -0.2, 1.3, 0.0])
    for tau in (1.0, 2.0):
        u = ph.stream_uniforms(5, traj=np.arange(n), step=1, stream=1, n=K)
        k, _, _ = wm.argmax_fp32(logits / tau + wm.gumbel(u), True)
        counts = np.bincount(k, minlength=K)
        res = stats.chisquare(counts, special.softmax(logits / tau) * n)
        assert res.pvalue > 1e-4


def test_box_muller_standard_normal_and_independent():
    u = ph.stream_uniforms(9, traj=np.arange(100000), step=0, stream=2, n=4)
    eps = wm.box_muller(u)
    for j in range(4):
        assert stats.kstest(eps[:, j], "norm").pvalue > 1e-4
    assert abs(np.corrcoef(eps[:, 0], eps[:, 1])[0, 1]) < 0.01
    assert abs(np.corrcoef(eps[:, 0], eps[:, 2])[0, 1]) < 0.01
    # the pair shares its radius: eps_2p^2 + eps_2p+1^2 = -2 ln u_2p
    np.testing.assert_allclose(eps[:, 0] ** 2 + eps[:, 1] ** 2, -2 * np.log(u[:, 0]), rtol=1e-12)


def test_single_component_sample_is_plain_normal():
    """K = 1: z' = mu + sigma * eps with eps a standard normal; checked by
    standardising many one-step samples with the oracle's own mu, sigma."""
    Z, H, A, K = 4, 6, 5, 1
    w = _weights(Z=Z, H=H, A=A, K=K)
    wb = wm.weight_blocks(w, Z, H, A, K, "fp32")
    n = 20000
    rng = np.random.default_rng(9)
    z = np.tile(rng.normal(size=(1, Z)), (n, 1))
    h = np.zeros((n, H))
    r = wm.transition(wb, dict(Z=Z, H=H, A=A, K=K), z, h, np.zeros((n, H)),
                      np.ones((n, A), np.uint8), seed=3, traj=np.arange(n), step=0,
                      done_flag=False, action=np.zeros(n, np.int64))
    zs = (r["z"] - r["mu"][..., 0]) / np.exp(r["log_sigma"][..., 0])
    for j in range(Z):
        assert stats.kstest(zs[:, j], "norm").pvalue > 1e-4
    assert np.all(r["component"] == 0)


# --------------------------------------------------------------------------
# rollout-level invariants
# --------------------------------------------------------------------------

def _rollout_case(B=12, T=6, Z=4, H=6, A=5, K=3, seed=7, dtype="fp32", mask_p=0.5):
    w = wl.Workload("t", "rollout", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype=dtype, seed=seed,
                    mask_p=mask_p)
    return w, wl.make_rollout_inputs(w)


def test_done_head_extremes_and_rate():
    w, d = _rollout_case(B=200, T=3)
    wts = dict(d["weights"])
    dims = w.dims
    wts["b_d"] = np.float32(30.0)
    r = wm.rollout(wts, dims, d["z0"], d["mask"], T=3, seed=1)
    assert np.all(r["dones"] == 1) and np.all(r["actions"][1:] == -1)
    assert np.all(r["actions"][0] >= 0)
    wts["b_d"] = np.float32(-30.0)
    r = wm.rollout(wts, dims, d["z0"], d["mask"], T=3, seed=1)
    assert np.all(r["dones"] == 0)
    # W_d = 0, b_d = logit(p): the done rate is p (binomial test)
    p = 0.2
    wts["w_d"] = np.zeros_like(wts["w_d"])
    wts["b_d"] = np.float32(math.log(p / (1 - p)))
    n = 4000
    z0 = np.zeros((n, w.Z), np.float32)
    r = wm.rollout(wts, dims, z0, np.ones((n, w.A), np.uint8), T=1, seed=2)
    assert stats.binomtest(int(r["dones"].sum()), n, p).pvalue > 1e-4


def test_masked_actions_never_taken_in_rollout():
    w, d = _rollout_case(B=64, T=8, mask_p=0.3)
    r = wm.rollout(d["weights"], w.dims, d["z0"], d["mask"], T=8, seed=3)
    a = r["actions"]
    taken = a >= 0
    rows = np.nonzero(taken)
    assert np.all(d["mask"][rows[1], a[taken]] == 1)


def test_empty_mask_row_ends_trajectory():
    w, d = _rollout_case(B=4, T=3)
    mask = d["mask"].copy()
    mask[2] = 0
    r = wm.rollout(d["weights"], w.dims, d["z0"], mask, T=3, seed=3, done_flag=False)
    assert r["actions"][:, 2].tolist() == [-1, -1, -1]
    assert r["dones"][:, 2].tolist() == [1, 1, 1]
    assert np.all(r["z_out"][:, 2] == d["z0"][2])
    assert r["done_T"][2] == 1


def test_resume_equals_single_rollout():
    w, d = _rollout_case(B=10, T=7)
    full = wm.rollout(d["weights"], w.dims, d["z0"], d["mask"], T=7, seed=5)
    a = wm.rollout(d["weights"], w.dims, d["z0"], d["mask"], T=3, seed=5)
    b = wm.rollout(d["weights"], w.dims, a["z_out"][-1], d["mask"], T=4, seed=5, step0=3,
                   h0=a["h_T"], c0=a["c_T"], done0=a["done_T"])
    np.testing.assert_array_equal(np.concatenate([a["actions"], b["actions"]]), full["actions"])
    np.testing.assert_array_equal(np.concatenate([a["dones"], b["dones"]]), full["dones"])
    np.testing.assert_allclose(np.concatenate([a["z_out"], b["z_out"][1:]]), full["z_out"],
                               rtol=0, atol=0)


def test_batch_subset_invariance():
    w, d = _rollout_case(B=16, T=5)
    full = wm.rollout(d["weights"], w.dims, d["z0"], d["mask"], T=5, seed=6)
    sub = wm.rollout(d["weights"], w.dims, d["z0"][5:11], d["mask"][5:11], T=5, seed=6, traj0=5)
    np.testing.assert_array_equal(sub["actions"], full["actions"][:, 5:11])
    np.testing.assert_array_equal(sub["z_out"], full["z_out"][:, 5:11])


def test_teacher_forcing_reproduces_rollout_state():
    """Feeding a rollout's own (z, a) to the NLL pass reproduces its h trace
    while all trajectories are live."""
    w, d = _rollout_case(B=8, T=5)
    r = wm.rollout(d["weights"], w.dims, d["z0"], d["mask"], T=5, seed=8, done_flag=False)
    assert np.all(r["actions"] >= 0)
    out = wm.nll(d["weights"], w.dims, r["z_out"], r["actions"], r["rewards"],
                 np.zeros((5, 8), np.uint8))
    np.testing.assert_allclose(out["h_trace"], r["h_trace"][1:], rtol=1e-13, atol=1e-14)
    # and the rollout's reward head equals the NLL pass's (se of its own reward is 0)
    np.testing.assert_allclose(out["reward_se"], 0.0, atol=1e-20)


def test_tau_scales_pi_logits_only():
    w, d = _rollout_case(B=6, T=1)
    wb = wm.weight_blocks(d["weights"], **w.dims, dtype="fp32")
    z, h, c = d["z0"].astype(np.float64), np.zeros((6, w.H)), np.zeros((6, w.H))
    kw = dict(seed=4, traj=np.arange(6), step=0, action=np.zeros(6, np.int64))
    r1 = wm.transition(wb, w.dims, z, h, c, d["mask"], tau=1.0, **kw)
    r2 = wm.transition(wb, w.dims, z, h, c, d["mask"], tau=2.5, **kw)
    np.testing.assert_array_equal(r1["mu"], r2["mu"])
    np.testing.assert_array_equal(r1["eps"], r2["eps"])
    # z' is mu + sigma eps of the component each temperature picked
    for r in (r1, r2):
        k = r["component"][..., None]
        ref = (np.take_along_axis(r["mu"], k, -1) + np.exp(np.take_along_axis(r["log_sigma"], k, -1))
               * r["eps"][..., None])[..., 0]
        np.testing.assert_array_equal(r["z"], ref)


def test_per_step_masks():
    """A [T, B, A] mask repeating the [B, A] one changes nothing; one-hot
    step masks force the action of every live step; masked actions are never
    taken under the step's own mask."""
    w, d = _rollout_case(B=10, T=5)
    kw = dict(T=w.T, seed=3, tau=1.0, done_flag=True, dtype="fp32")
    ref = wm.rollout(d["weights"], w.dims, d["z0"], d["mask"], **kw)
    rep = wm.rollout(d["weights"], w.dims, d["z0"], np.broadcast_to(d["mask"], (w.T,) + d["mask"].shape), **kw)
    for k in ("z_out", "actions", "rewards", "dones"):
        np.testing.assert_array_equal(ref[k], rep[k])
    rng = np.random.default_rng(4)
    forced = rng.integers(0, w.A, size=(w.T, w.B))
    onehot = np.zeros((w.T, w.B, w.A), np.uint8)
    np.put_along_axis(onehot, forced[..., None], 1, axis=-1)
    r = wm.rollout(d["weights"], w.dims, d["z0"], onehot, **kw)
    live = r["actions"] >= 0
    assert live[0].all()
    np.testing.assert_array_equal(r["actions"][live], forced[live])
    sm = (rng.random((w.T, w.B, w.A)) < 0.5).astype(np.uint8)
    sm[..., 0] = 1
    r = wm.rollout(d["weights"], w.dims, d["z0"], sm, **kw)
    tt, bb = np.nonzero(r["actions"] >= 0)
    assert np.all(sm[tt, bb, r["actions"][tt, bb]] == 1)


def test_sigma_tau_scales_the_spread_only():
    """With sigma_tau the draw is mu + sqrt(tau) sigma eps: at tau = 1 nothing
    changes; at tau = 2.25 the component picks, means and eps stay, and with
    K = 1 many one-step samples standardised by 1.5 sigma are standard normal."""
    w, d = _rollout_case(B=6, T=1)
    wb = wm.weight_blocks(d["weights"], **w.dims, dtype="fp32")
    z, h, c = d["z0"].astype(np.float64), np.zeros((6, w.H)), np.zeros((6, w.H))
    kw = dict(seed=4, traj=np.arange(6), step=0, action=np.zeros(6, np.int64))
    r0 = wm.transition(wb, w.dims, z, h, c, d["mask"], tau=1.0, **kw)
    r1 = wm.transition(wb, w.dims, z, h, c, d["mask"], tau=1.0, sigma_tau=True, **kw)
    np.testing.assert_array_equal(r0["z"], r1["z"])
    a = wm.transition(wb, w.dims, z, h, c, d["mask"], tau=2.25, **kw)
    b = wm.transition(wb, w.dims, z, h, c, d["mask"], tau=2.25, sigma_tau=True, **kw)
    np.testing.assert_array_equal(a["component"], b["component"])
    k = a["component"][..., None]
    mu_k = np.take_along_axis(a["mu"], k, -1)[..., 0]
    np.testing.assert_allclose(b["z"] - mu_k, 1.5 * (a["z"] - mu_k), rtol=1e-12, atol=1e-12)

    Z, H, A, K = 4, 6, 5, 1
    w1 = _weights(Z=Z, H=H, A=A, K=K)
    wb1 = wm.weight_blocks(w1, Z, H, A, K, "fp32")
    n = 20000
    rng = np.random.default_rng(11)
    zz = np.tile(rng.normal(size=(1, Z)), (n, 1))
    r = wm.transition(wb1, dict(Z=Z, H=H, A=A, K=K), zz, np.zeros((n, H)), np.zeros((n, H)),
                      np.ones((n, A), np.uint8), seed=5, traj=np.arange(n), step=0, tau=2.25,
                      done_flag=False, action=np.zeros(n, np.int64), sigma_tau=True)
    zs = (r["z"] - r["mu"][..., 0]) / (1.5 * np.exp(r["log_sigma"][..., 0]))
    for j in range(Z):
        assert stats.kstest(zs[:, j], "norm").pvalue > 1e-4


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_workload_generators_deterministic(dtype):
    w = wl.Workload("t", "rollout", B=8, T=4, Z=8, H=16, A=6, K=2, dtype=dtype, seed=3)
    a, b = wl.make_rollout_inputs(w), wl.make_rollout_inputs(w)
    for k in ("z0", "mask"):
        np.testing.assert_array_equal(a[k], b[k])
    assert np.all(a["mask"].sum(1) >= 1)
    n = wl.make_nll_inputs(w.replace(kind="nll"))
    assert np.all(n["mask"][np.arange(8)[None, :].repeat(4, 0), n["actions"]] == 1)
