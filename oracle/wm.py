"""Vectorised float64 oracle of the World-Model dream rollout and NLL pass.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The method (RLFlow, arXiv 2205.01435):
* section 3.3.2 (MDN-RNN): a recurrent network over the latent z_t and the
  action a_t models P(z_{t+1} | a_t, z_t, h_t); its outputs parameterise a
  Gaussian mixture whose weights pi come from a softmax of logits divided by
  a temperature tau; z_{t+1} is drawn from that mixture.
* section 3.4 (Action Controller): a_t = W_c [z_t, h_t] + b_c, read here as
  action logits.
* section 3.1.3 (State-Action space): invalid actions are masked out of the
  logits so that only valid actions can be chosen.
* section 3.1.1 (System environment): a step returns the next state, a
  reward and a terminal flag.
* section 3.3.1 (Recurrent Neural Networks): padded sequences are masked.

Readings where the paper is silent (each also listed in the design notes):
LSTM cell, gate order (i, f, g, o), one bias, no peepholes; one independent
K-component 1-D mixture per latent dimension; sigma = exp(log sigma);
tau > 0 divides the pi-logits only; categorical draws by Gumbel-max on
Philox uniforms (ties to the lowest index, decided on float32-rounded scores
as the device decides them); Gaussian draws by Box-Muller on dimension pairs
(2p, 2p+1); reward and done heads read h_{t+1}; done = sigmoid(rho_d) > u;
a finished trajectory freezes; the one-hot action enters the gates as a
column of the action block of W_g.

Precision: float64 throughout.  On bf16 workloads ``q`` rounds weights, the
GEMM operands z and h, and the stored h to bfloat16 (the device's rounding
points); c, logits and mixture arithmetic stay at full precision.
"""

from __future__ import annotations

import math

import numpy as np
from scipy.special import expit

from . import philox as ph
from .bf16 import q

LN_2PI = math.log(2.0 * math.pi)


# ----------------------------------------------------------------------------
# weights
# ----------------------------------------------------------------------------

def weight_blocks(w: dict, Z: int, H: int, A: int, K: int, dtype: str) -> dict:
    """Storage-rounded float64 weight blocks.

    W_g columns are z | one-hot a | h; its action block holds one column per
    action (the one-hot input selects a column, section 3.3.2's a_t input).
    """
    Wg = q(w["W_g"], dtype)
    if Wg.shape != (4 * H, Z + A + H):
        raise ValueError(f"W_g shape {Wg.shape} != {(4 * H, Z + A + H)}")
    return dict(
        Wz=Wg[:, :Z], Wa=Wg[:, Z:Z + A], Wh=Wg[:, Z + A:],
        b_g=np.asarray(w["b_g"], np.float64),
        W_m=q(w["W_m"], dtype), b_m=np.asarray(w["b_m"], np.float64),
        w_r=q(w["w_r"], dtype), b_r=float(np.asarray(w["b_r"]).reshape(-1)[0]),
        w_d=q(w["w_d"], dtype), b_d=float(np.asarray(w["b_d"]).reshape(-1)[0]),
        W_c=q(w["W_c"], dtype), b_c=np.asarray(w["b_c"], np.float64),
    )


# ----------------------------------------------------------------------------
# building blocks
# ----------------------------------------------------------------------------

def gumbel(u) -> np.ndarray:
    """Standard Gumbel variate -ln(-ln u) of a uniform u in (0, 1)."""
    return -np.log(-np.log(u))


def argmax_fp32(scores, valid):
    """Gumbel-max decision.

    Returns ``(index, margin, top)``: the index of the largest score among the
    valid entries after rounding the scores to float32 (the device's
    precision), the lowest index on ties and -1 when no entry is valid; the
    float64 gap between the best and second-best valid score (inf when fewer
    than two are valid); and the best float64 score.
    """
    scores = np.asarray(scores, np.float64)
    valid = np.broadcast_to(np.asarray(valid, bool), scores.shape)
    s32 = np.where(valid, scores.astype(np.float32), np.float32(-np.inf))
    idx = np.argmax(s32, axis=-1)  # first occurrence of the maximum
    has = valid.any(axis=-1)
    idx = np.where(has, idx, -1)
    s64 = np.where(valid, scores, -np.inf)
    if scores.shape[-1] >= 2:
        top2 = np.sort(s64, axis=-1)[..., -2:]
        top, second = top2[..., 1], top2[..., 0]
        with np.errstate(invalid="ignore"):
            margin = np.where(np.isfinite(second), top - second, np.inf)
    else:
        top = s64[..., 0]
        margin = np.full(top.shape, np.inf)
    return idx.astype(np.int64), margin, top


def controller_logits(wb: dict, z, h, dtype: str) -> np.ndarray:
    """Section 3.4: logits = W_c [z_t, h_t] + b_c on the storage-rounded state."""
    x = np.concatenate([q(z, dtype), q(h, dtype)], axis=-1)
    return x @ wb["W_c"].T + wb["b_c"]


def two_level_action(logits, xmask, lmask, *, seed: int, traj, step: int, N: int, L: int,
                     return_xfer: bool = False):
    """The two-level action of section 3.1.3: the controller first picks a
    graph transformation (xfer) among the valid ones, index N being the NO-OP
    that ends the episode, then a location among those valid for that xfer.

    ``logits [n, N+1+L]``: xfer logits (N+1) then location logits (L), from
    the same controller input; ``xmask [n, N+1]``, ``lmask [n, N, L]``.
    Each pick is a Gumbel-max (xfers on stream 0, index x; locations on
    stream 4, index l).  Returns ``(a, margin, top)``: the flat action
    a = x L + l of the world model's one-hot input, -2 for the NO-OP, -1 when
    no xfer (or no location of the chosen xfer) is valid; and the margin and
    top score of the pick with the smaller relative margin, for near-tie
    checks (and, with ``return_xfer``, the picked xfer: N for the NO-OP, -1
    when none is valid).
    """
    logits = np.asarray(logits, np.float64)
    n = logits.shape[0]
    xmask = np.asarray(xmask) != 0
    lmask = np.asarray(lmask) != 0
    u0 = ph.stream_uniforms(seed, traj, step, ph.STREAM_CONTROLLER, N + 1)
    x, xm, xt = argmax_fp32(logits[:, :N + 1] + gumbel(u0), xmask)
    u4 = ph.stream_uniforms(seed, traj, step, ph.STREAM_LOCATION, L)
    rows = lmask[np.arange(n), np.clip(x, 0, max(N - 1, 0))]
    loc, lm, lt = argmax_fp32(logits[:, N + 1:] + gumbel(u4), rows)
    xfer = (x >= 0) & (x < N)
    a = np.where(x < 0, -1, np.where(x == N, -2, np.where(loc < 0, -1, x * L + loc)))
    with np.errstate(invalid="ignore"):
        use_l = xfer & (lm / (1 + np.abs(lt)) < xm / (1 + np.abs(xt)))
    out = (a.astype(np.int64), np.where(use_l, lm, xm), np.where(use_l, lt, xt))
    return out + (x,) if return_xfer else out


def masked_softmax(logits, mask) -> np.ndarray:
    """Softmax over the valid actions only (section 3.1.3 masks invalid
    logits); masked entries are exactly 0, an all-invalid row is all 0."""
    logits = np.asarray(logits, np.float64)
    valid = np.asarray(mask) != 0
    m = np.max(np.where(valid, logits, -np.inf), axis=-1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(valid, np.exp(np.where(valid, logits - m, 0.0)), 0.0)
    s = e.sum(axis=-1, keepdims=True)
    return np.where(s > 0, e / np.where(s > 0, s, 1.0), 0.0)


def gate_preactivations(wb: dict, z, h, a, dtype: str) -> np.ndarray:
    """Gate pre-activations g = W_z z + W_h h + W_a onehot(a) + b_g.

    The one-hot product is the column ``W_a[:, a]``; an action outside
    ``[0, A)`` (no action) contributes the zero vector.
    """
    g = q(z, dtype) @ wb["Wz"].T + q(h, dtype) @ wb["Wh"].T + wb["b_g"]
    a = np.asarray(a, np.int64)
    A = wb["Wa"].shape[1]
    ok = (a >= 0) & (a < A)
    g = g + np.where(ok[:, None], wb["Wa"][:, np.where(ok, a, 0)].T, 0.0)
    return g


def lstm_cell(g, c):
    """LSTM cell on pre-activations ``g [N, 4H]`` (gate blocks i | f | g | o):
    c' = sigma(f) c + sigma(i) tanh(g),  h' = sigma(o) tanh(c')."""
    H = g.shape[-1] // 4
    i = expit(g[..., 0:H])
    f = expit(g[..., H:2 * H])
    gg = np.tanh(g[..., 2 * H:3 * H])
    o = expit(g[..., 3 * H:4 * H])
    c2 = f * c + i * gg
    h2 = o * np.tanh(c2)
    return h2, c2


def mdn_params(wb: dict, h_next, Z: int, K: int, dtype: str):
    """Mixture parameters from h_{t+1} (section 3.3.2): per latent dim j and
    component k the pi-logit, mean and log standard deviation, each
    ``[N, Z, K]`` (W_m row p*Z*K + j*K + k)."""
    m = q(h_next, dtype) @ wb["W_m"].T + wb["b_m"]
    m = m.reshape(m.shape[0], 3, Z, K)
    return m[:, 0], m[:, 1], m[:, 2]


def reward_done_logits(wb: dict, h_next, dtype: str):
    """Reward and done heads on h_{t+1}: rho_r = w_r . h + b_r, rho_d = w_d . h + b_d."""
    hq = q(h_next, dtype)
    return hq @ wb["w_r"] + wb["b_r"], hq @ wb["w_d"] + wb["b_d"]


def mixture_weights(logit_pi, tau: float) -> np.ndarray:
    """Temperature softmax of section 3.3.2: exp(x_k / tau) / sum_j exp(x_j / tau)."""
    x = np.asarray(logit_pi, np.float64) / tau
    x = x - x.max(axis=-1, keepdims=True)
    e = np.exp(x)
    return e / e.sum(axis=-1, keepdims=True)


def box_muller(u) -> np.ndarray:
    """Standard normals from uniforms ``u [..., Z]`` (Z even): for each pair
    (2p, 2p+1), r = sqrt(-2 ln u_2p), theta = 2 pi u_2p+1, eps_2p = r cos theta,
    eps_2p+1 = r sin theta."""
    u = np.asarray(u, np.float64)
    r = np.sqrt(-2.0 * np.log(u[..., 0::2]))
    th = 2.0 * np.pi * u[..., 1::2]
    eps = np.empty(u.shape, np.float64)
    eps[..., 0::2] = r * np.cos(th)
    eps[..., 1::2] = r * np.sin(th)
    return eps


def log_softmax(x, axis=-1):
    m = np.max(x, axis=axis, keepdims=True)
    return x - (m + np.log(np.sum(np.exp(x - m), axis=axis, keepdims=True)))


def logsumexp(x, axis=-1):
    """max + log sum exp(x - max)."""
    m = np.max(x, axis=axis, keepdims=True)
    return (m + np.log(np.sum(np.exp(x - m), axis=axis, keepdims=True))).squeeze(axis)


def softplus(x):
    x = np.asarray(x, np.float64)
    return np.maximum(x, 0.0) + np.log1p(np.exp(-np.abs(x)))


# ----------------------------------------------------------------------------
# one dream transition
# ----------------------------------------------------------------------------

def transition(wb: dict, dims: dict, z, h, c, mask, *, seed: int, traj, step: int,
               tau: float = 1.0, done_flag: bool = True, dtype: str = "fp32",
               action=None, h_next=None, sigma_tau: bool = False, two_level=None) -> dict:
    """One dream step for a batch of live rows (sections 3.4 and 3.3.2).

    1. controller logits on [z_t, h_t] and a masked Gumbel-max action
       (stream 0; no valid action -> -1);
    2. gates W_z z + W_h h + W_a[:, a] + b_g and the LSTM cell -> h', c';
    3. mixture parameters and reward/done logits from h' (or from
       ``h_next`` when given, to re-anchor on another implementation's h');
    4. per latent dim a Gumbel-max component pick on pi-logit / tau (stream 1);
    5. z'_j = mu_{j,k} + exp(log sigma_{j,k}) eps_j, eps from Box-Muller on
       stream 2 (with ``sigma_tau`` the standard deviation is also scaled by
       sqrt(tau), the temperature of Ha and Schmidhuber's World Models, whose
       model section 3.3 builds on; the paper itself applies tau to pi only);
    6. reward = rho_r; done = sigmoid(rho_d) > u (stream 3) when enabled.

    ``action`` overrides the controller's choice in step 2 (re-anchoring).
    With ``two_level = (N, L)`` the controller is the two-level one of
    ``two_level_action`` and ``mask`` is the pair (xfer mask, location mask).
    """
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    z = np.asarray(z, np.float64)
    h = np.asarray(h, np.float64)
    c = np.asarray(c, np.float64)
    traj = np.asarray(traj, np.int64)
    n = z.shape[0]

    logits = controller_logits(wb, z, h, dtype)
    if two_level is not None:
        a, a_margin, a_top = two_level_action(logits, mask[0], mask[1], seed=seed, traj=traj,
                                              step=step, N=two_level[0], L=two_level[1])
    else:
        u0 = ph.stream_uniforms(seed, traj, step, ph.STREAM_CONTROLLER, A)
        a, a_margin, a_top = argmax_fp32(logits + gumbel(u0), np.asarray(mask) != 0)
    a_used = a if action is None else np.asarray(action, np.int64)

    g = gate_preactivations(wb, z, h, a_used, dtype)
    h2, c2 = lstm_cell(g, c)
    h2 = q(h2, dtype)
    hh = h2 if h_next is None else q(h_next, dtype)

    logit_pi, mu, log_sigma = mdn_params(wb, hh, Z, K, dtype)
    rho_r, rho_d = reward_done_logits(wb, hh, dtype)

    u1 = ph.stream_uniforms(seed, traj, step, ph.STREAM_COMPONENT, Z * K).reshape(n, Z, K)
    k, k_margin, k_top = argmax_fp32(logit_pi / tau + gumbel(u1), True)
    u2 = ph.stream_uniforms(seed, traj, step, ph.STREAM_GAUSS, Z)
    eps = box_muller(u2)
    mu_k = np.take_along_axis(mu, k[..., None], axis=-1)[..., 0]
    ls_k = np.take_along_axis(log_sigma, k[..., None], axis=-1)[..., 0]
    z2 = mu_k + np.exp(ls_k) * (math.sqrt(tau) * eps if sigma_tau else eps)

    if done_flag:
        u3 = ph.stream_uniforms(seed, traj, step, ph.STREAM_DONE, 1)[:, 0]
        p_done = expit(rho_d)
        d = p_done.astype(np.float32) > u3.astype(np.float32)
        d_margin = np.abs(p_done - u3)
    else:
        d = np.zeros(n, bool)
        d_margin = np.full(n, np.inf)

    return dict(action=a, action_margin=a_margin, action_top=a_top, logits=logits,
                gates=g, h=h2, c=c2, logit_pi=logit_pi, mu=mu, log_sigma=log_sigma,
                component=k, component_margin=k_margin, component_top=k_top,
                eps=eps, z=z2, reward=rho_r, done_logit=rho_d, done=d,
                done_margin=d_margin)


# ----------------------------------------------------------------------------
# entry points
# ----------------------------------------------------------------------------

def rollout(w: dict, dims: dict, z0, mask, *, T: int, seed: int, tau: float = 1.0,
            done_flag: bool = True, dtype: str = "fp32", traj0: int = 0, step0: int = 0,
            h0=None, c0=None, done0=None, sigma_tau: bool = False, two_level=None,
            lengths=None) -> dict:
    """B dream trajectories of T steps (the "hallucinated" environment of
    section 3.3 driven by the controller of section 3.4).

    Transition t uses absolute step s = step0 + t and trajectory index
    traj0 + b for its random streams.  A trajectory that is done (input flag,
    a sampled done, or no valid action) is frozen afterwards: action -1,
    reward 0, done 1, z copied, state (z, h, c) unchanged.  A row with no
    valid action ends at that step with the same frozen outputs.  ``mask`` is
    [B, A] for every step, or [T, B, A] with one mask per step (the valid
    actions depend on the state, section 3.1.3).  With ``two_level = (N, L)``
    the controller is two-level (``two_level_action``), ``mask`` is the pair
    (xfer mask [B, N+1], location mask [B, N, L]) and a NO-OP ends the
    trajectory with action -2 at that step.

    ``lengths [B]`` (optional) gives each trajectory its own horizon, as
    variable-length sequences are zero-padded and masked (section 3.3.1):
    trajectory b is stepped for t < lengths[b] only; a step t >= lengths[b]
    is padding, with action -1, reward 0, done 0 and z_out[t+1] = 0, and the
    state stays as it was after step lengths[b] - 1 (h_T, c_T, done_T are
    that state).

    Returns z_out [T+1, B, Z], actions [T, B], rewards [T, B], dones [T, B],
    h_T, c_T [B, H], done_T [B], the state trace h_trace, c_trace [T+1, B, H]
    (state at the start of each step) and the decision margins
    (action_margin [T, B], component_margin [T, B, Z], done_margin [T, B];
    NaN where frozen).
    """
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    wb = weight_blocks(w, Z, H, A, K, dtype)
    z0 = np.asarray(z0, np.float64)
    B = z0.shape[0]
    if two_level is None:
        mask = np.asarray(mask)
    z = z0.copy()
    h = np.zeros((B, H)) if h0 is None else q(h0, dtype)
    c = np.zeros((B, H)) if c0 is None else np.asarray(c0, np.float64).copy()
    done = np.zeros(B, bool) if done0 is None else np.asarray(done0) != 0

    z_out = np.empty((T + 1, B, Z))
    z_out[0] = z
    actions = np.full((T, B), -1, np.int32)
    rewards = np.zeros((T, B))
    dones = np.ones((T, B), np.uint8)
    h_trace = np.empty((T + 1, B, H))
    c_trace = np.empty((T + 1, B, H))
    a_margin = np.full((T, B), np.nan)
    k_margin = np.full((T, B, Z), np.nan)
    d_margin = np.full((T, B), np.nan)

    horizon = np.full(B, T, np.int64) if lengths is None else np.clip(np.asarray(lengths, np.int64), 0, T)
    for t in range(T):
        h_trace[t], c_trace[t] = h, c
        live = np.nonzero(~done & (t < horizon))[0]
        if live.size:
            if two_level is not None:
                mask_l = (np.asarray(mask[0])[live], np.asarray(mask[1])[live])
            else:
                mask_t = mask[t] if mask.ndim == 3 else mask  # per-step masks: [T, B, A]
                mask_l = mask_t[live]
            r = transition(wb, dims, z[live], h[live], c[live], mask_l, seed=seed,
                           traj=traj0 + live, step=step0 + t, tau=tau,
                           done_flag=done_flag, dtype=dtype, sigma_tau=sigma_tau,
                           two_level=two_level)
            ok = r["action"] >= 0
            a_margin[t, live] = r["action_margin"]
            rows = live[ok]
            actions[t, rows] = r["action"][ok]
            rewards[t, rows] = r["reward"][ok]
            dones[t, rows] = r["done"][ok].astype(np.uint8)
            k_margin[t, rows] = r["component_margin"][ok]
            d_margin[t, rows] = r["done_margin"][ok]
            z[rows] = r["z"][ok]
            h[rows] = r["h"][ok]
            c[rows] = r["c"][ok]
            done[rows] = r["done"][ok]
            done[live[~ok]] = True
            actions[t, live[r["action"] == -2]] = -2  # the NO-OP ended these
        z_out[t + 1] = z
        pad = t >= horizon  # padding: zero latent, no action, reward 0, not done
        z_out[t + 1, pad] = 0.0
        dones[t, pad] = 0
    h_trace[T], c_trace[T] = h, c
    return dict(z_out=z_out, actions=actions, rewards=rewards, dones=dones,
                h_T=h.copy(), c_T=c.copy(), done_T=done.astype(np.uint8),
                h_trace=h_trace, c_trace=c_trace, action_margin=a_margin,
                component_margin=k_margin, done_margin=d_margin)


def controller_step(w: dict, dims: dict, z, h, mask, *, seed: int, step: int,
                    traj0: int = 0, dtype: str = "fp32", two_level=None) -> dict:
    """One controller decision (section 3.4 with the masking of section 3.1.3):
    masked softmax probabilities of the logits (tau = 1) and a Gumbel-max
    sample from them on stream 0 of (seed, traj0 + b, step).

    With ``two_level = (N, L)`` (section 3.1.3's xfer, then location) and
    ``mask`` the pair (xfer mask [B, N+1], location mask [B, N, L]): the
    action of ``two_level_action`` and ``probs [B, N+1+L]``, the masked
    softmax of the xfer logits followed by the masked softmax of the location
    logits over the locations valid for the picked xfer (all 0 when the NO-OP
    or nothing was picked)."""
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    wb = weight_blocks(w, Z, H, A, K, dtype)
    z = np.asarray(z, np.float64)
    B = z.shape[0]
    logits = controller_logits(wb, z, h, dtype)
    traj = traj0 + np.arange(B)
    if two_level is not None:
        N, L = two_level
        xm, lm = np.asarray(mask[0]) != 0, np.asarray(mask[1]) != 0
        a, margin, top, x = two_level_action(logits, xm, lm, seed=seed, traj=traj, step=step, N=N, L=L,
                                             return_xfer=True)
        chosen = (x >= 0) & (x < N)
        lrow = np.where(chosen[:, None], lm[np.arange(B), np.clip(x, 0, N - 1)], False)
        probs = np.concatenate([masked_softmax(logits[:, :N + 1], xm),
                                masked_softmax(logits[:, N + 1:], lrow)], axis=1)
        return dict(probs=probs, action=a.astype(np.int32), margin=margin, top=top, logits=logits,
                    xfer=x)
    u0 = ph.stream_uniforms(seed, traj, step, ph.STREAM_CONTROLLER, A)
    a, margin, top = argmax_fp32(logits + gumbel(u0), np.asarray(mask) != 0)
    return dict(probs=masked_softmax(logits, mask), action=a.astype(np.int32),
                margin=margin, top=top, logits=logits)


def nll(w: dict, dims: dict, z, actions, rewards, dones, *, lengths=None,
        dtype: str = "fp32") -> dict:
    """Teacher-forced MDN-RNN loss over logged sequences (the log-likelihood
    loss of section 4.7, fitted on random-agent rollouts, section 3.3.2).

    For each sequence b and step t < len[b], with h_0 = c_0 = 0:
      h_{t+1}, c_{t+1} = LSTM(W_z z_t + W_h h_t + W_a[:, a_t] + b_g, c_t);
      loglik[t, b] = sum_j log sum_k pi_jk N(z_{t+1,j}; mu_jk, sigma_jk)
                   (pi at tau = 1);
      reward_se[t, b] = (rho_r - r_t)^2;
      done_bce[t, b] = softplus(rho_d) - d_t rho_d;
    steps t >= len[b] are padding (section 3.3.1) and output 0.
    means = (-sum loglik / (N Z), sum se / N, sum bce / N), N = sum len.
    """
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    wb = weight_blocks(w, Z, H, A, K, dtype)
    z = np.asarray(z, np.float64)
    actions = np.asarray(actions, np.int64)
    T, B = actions.shape
    lengths = np.full(B, T, np.int64) if lengths is None else np.asarray(lengths, np.int64)
    lengths = np.clip(lengths, 0, T)
    h = np.zeros((B, H))
    c = np.zeros((B, H))
    h_next = np.empty((T, B, H))
    for t in range(T):
        g = gate_preactivations(wb, z[t], h, actions[t], dtype)
        h2, c = lstm_cell(g, c)
        h = q(h2, dtype)
        h_next[t] = h
    hf = h_next.reshape(T * B, H)
    logit_pi, mu, log_sigma = mdn_params(wb, hf, Z, K, dtype)
    target = z[1:].reshape(T * B, Z)[..., None]
    log_pi = log_softmax(logit_pi, axis=-1)
    log_n = -0.5 * ((target - mu) / np.exp(log_sigma)) ** 2 - log_sigma - 0.5 * LN_2PI
    ll = logsumexp(log_pi + log_n, axis=-1).sum(axis=-1).reshape(T, B)
    rho_r, rho_d = reward_done_logits(wb, hf, dtype)
    se = (rho_r.reshape(T, B) - np.asarray(rewards, np.float64)) ** 2
    dd = np.asarray(dones, np.float64)
    bce = softplus(rho_d.reshape(T, B)) - dd * rho_d.reshape(T, B)
    valid = np.arange(T)[:, None] < lengths[None, :]
    ll = np.where(valid, ll, 0.0)
    se = np.where(valid, se, 0.0)
    bce = np.where(valid, bce, 0.0)
    N = int(lengths.sum())
    if N > 0:
        means = np.array([-ll.sum() / (N * Z), se.sum() / N, bce.sum() / N])
    else:
        means = np.zeros(3)
    return dict(loglik=ll, reward_se=se, done_bce=bce, means=means, h_trace=h_next)
