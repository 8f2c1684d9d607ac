"""Float64 oracle of one world-model training step: the gradient of the
teacher-forced loss and the optimiser update.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The world model is fitted on the log-likelihood loss of section 4.7 (on
random-agent data, section 3.3.2), with the learning rate decayed over 5000
epochs by a second-degree polynomial (section 4.7's training curves).

Readings (also listed in the design notes):
* the loss is the sum of the three means of the NLL pass,
      L = -sum loglik / (N Z) + sum se / N + sum bce / N,
  so that the reward and done heads are fitted next to the mixture;
* the parameters are W_g, b_g, W_m, b_m, w_r, b_r, w_d, b_d (the
  controller is not part of the world model's loss); z, actions, rewards
  and dones are data;
* the optimiser is Adam (beta1 0.9, beta2 0.999, eps 1e-8), which the paper
  does not name; the learning rate at epoch e is
      (lr0 - lr_end) (1 - min(e, E) / E)^2 + lr_end,  E = 5000;
* fp32 weights (the NLL workload's precision).

The gradient is written out by hand (backpropagation through time through
the LSTM and the mixture, reward and done heads), step by step in the
forward pass's notation; ``tests/test_oracle_train.py`` pins it against
central finite differences of ``oracle.wm.nll``.
"""

from __future__ import annotations

import numpy as np
from scipy.special import expit

from . import wm

PARAMS = ("W_g", "b_g", "W_m", "b_m", "w_r", "b_r", "w_d", "b_d")


def loss(w: dict, dims: dict, z, actions, rewards, dones, lengths=None) -> float:
    """The summed means of the NLL pass (the training loss)."""
    m = wm.nll(w, dims, z, actions, rewards, dones, lengths=lengths)["means"]
    return float(m.sum())


def loss_and_grads(w: dict, dims: dict, z, actions, rewards, dones, lengths=None):
    """(loss, {param: gradient}) of the training loss, float64."""
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    Wg = np.asarray(w["W_g"], np.float64)
    Wz, Wa, Wh = Wg[:, :Z], Wg[:, Z:Z + A], Wg[:, Z + A:]
    bg = np.asarray(w["b_g"], np.float64)
    Wm = np.asarray(w["W_m"], np.float64)
    bm = np.asarray(w["b_m"], np.float64)
    wr = np.asarray(w["w_r"], np.float64)
    wd = np.asarray(w["w_d"], np.float64)
    br = float(np.asarray(w["b_r"]).reshape(-1)[0])
    bd = float(np.asarray(w["b_d"]).reshape(-1)[0])
    z = np.asarray(z, np.float64)
    actions = np.asarray(actions, np.int64)
    T, B = actions.shape
    lengths = np.full(B, T, np.int64) if lengths is None else np.clip(np.asarray(lengths, np.int64), 0, T)
    valid = (np.arange(T)[:, None] < lengths[None, :]).astype(np.float64)
    N = int(lengths.sum())
    if N == 0:
        return 0.0, {k: np.zeros_like(np.asarray(w[k], np.float64)) for k in PARAMS}

    # forward, keeping what the backward pass needs
    onehot = np.zeros((T, B, A))
    ok = (actions >= 0) & (actions < A)
    tt, bb = np.nonzero(ok)
    onehot[tt, bb, actions[tt, bb]] = 1.0
    h = np.zeros((T + 1, B, H))
    c = np.zeros((T + 1, B, H))
    gi, gf, gg, go = (np.zeros((T, B, H)) for _ in range(4))
    for t in range(T):
        g = z[t] @ Wz.T + onehot[t] @ Wa.T + h[t] @ Wh.T + bg
        gi[t], gf[t] = expit(g[:, :H]), expit(g[:, H:2 * H])
        gg[t], go[t] = np.tanh(g[:, 2 * H:3 * H]), expit(g[:, 3 * H:])
        c[t + 1] = gf[t] * c[t] + gi[t] * gg[t]
        h[t + 1] = go[t] * np.tanh(c[t + 1])

    # heads on h_{t+1}
    hn = h[1:]                                       # [T, B, H]
    m = hn @ Wm.T + bm                               # [T, B, 3ZK]
    m3 = m.reshape(T, B, 3, Z, K)
    lpi_logit, mu, ls = m3[:, :, 0], m3[:, :, 1], m3[:, :, 2]
    x = z[1:][..., None]                             # [T, B, Z, 1] targets
    log_pi = wm.log_softmax(lpi_logit, axis=-1)
    sig = np.exp(ls)
    u = (x - mu) / sig
    log_n = -0.5 * u ** 2 - ls - 0.5 * wm.LN_2PI
    joint = log_pi + log_n
    ll = wm.logsumexp(joint, axis=-1)                 # [T, B, Z]
    gam = np.exp(joint - ll[..., None])               # responsibilities
    pi = np.exp(log_pi)
    rho_r = hn @ wr + br
    rho_d = hn @ wd + bd
    r = np.asarray(rewards, np.float64)
    dn = np.asarray(dones, np.float64)
    L = (-(ll.sum(-1) * valid).sum() / (N * Z) + (((rho_r - r) ** 2) * valid).sum() / N
         + ((wm.softplus(rho_d) - dn * rho_d) * valid).sum() / N)

    # d L / d head outputs
    s_ll = -valid[..., None, None] / (N * Z)         # d L / d loglik_j
    d_lpi = s_ll * (gam - pi)                         # through log_softmax and the LSE
    d_mu = s_ll * gam * u / sig
    d_ls = s_ll * gam * (u ** 2 - 1.0)
    dm = np.stack([d_lpi, d_mu, d_ls], axis=2).reshape(T, B, 3 * Z * K)
    d_rr = 2.0 * (rho_r - r) * valid / N
    d_rd = (expit(rho_d) - dn) * valid / N

    grads = {
        "W_m": np.einsum("tbn,tbh->nh", dm, hn),
        "b_m": dm.sum(axis=(0, 1)),
        "w_r": np.einsum("tb,tbh->h", d_rr, hn),
        "b_r": np.array([d_rr.sum()]),
        "w_d": np.einsum("tb,tbh->h", d_rd, hn),
        "b_d": np.array([d_rd.sum()]),
    }
    dh_head = dm @ Wm + d_rr[..., None] * wr + d_rd[..., None] * wd   # d L / d h_{t+1} from the heads

    # backpropagation through time
    dWz, dWa, dWh = np.zeros_like(Wz), np.zeros_like(Wa), np.zeros_like(Wh)
    dbg = np.zeros_like(bg)
    dh_next = np.zeros((B, H))   # d L / d h_{t+1} through step t+1
    dc_next = np.zeros((B, H))   # d L / d c_{t+1} through step t+1
    for t in range(T - 1, -1, -1):
        dh = dh_head[t] + dh_next
        th = np.tanh(c[t + 1])
        d_o = dh * th
        dc = dc_next + dh * go[t] * (1.0 - th ** 2)
        d_i = dc * gg[t]
        d_f = dc * c[t]
        d_g = dc * gi[t]
        dG = np.concatenate([d_i * gi[t] * (1 - gi[t]), d_f * gf[t] * (1 - gf[t]),
                             d_g * (1 - gg[t] ** 2), d_o * go[t] * (1 - go[t])], axis=1)  # [B, 4H]
        dWz += dG.T @ z[t]
        dWa += dG.T @ onehot[t]
        dWh += dG.T @ h[t]
        dbg += dG.sum(axis=0)
        dh_next = dG @ Wh
        dc_next = dc * gf[t]
    grads["W_g"] = np.concatenate([dWz, dWa, dWh], axis=1)
    grads["b_g"] = dbg
    return L, grads


def poly_lr(epoch: int, lr0: float, lr_end: float, epochs: int = 5000, power: float = 2.0) -> float:
    """Second-degree polynomial decay from lr0 to lr_end over `epochs`."""
    e = min(max(epoch, 0), epochs)
    return (lr0 - lr_end) * (1.0 - e / epochs) ** power + lr_end


def adam_step(params: dict, grads: dict, state: dict, lr: float, beta1: float = 0.9,
              beta2: float = 0.999, eps: float = 1e-8) -> dict:
    """One Adam update (Kingma and Ba, 2015) with bias correction; ``state``
    holds the moments m, v per parameter and the step count t (updated in
    place).  Returns the new parameters."""
    t = state.get("t", 0) + 1
    state["t"] = t
    out = {}
    for k, g in grads.items():
        g = np.asarray(g, np.float64)
        m = beta1 * state.get("m_" + k, np.zeros_like(g)) + (1 - beta1) * g
        v = beta2 * state.get("v_" + k, np.zeros_like(g)) + (1 - beta2) * g * g
        state["m_" + k], state["v_" + k] = m, v
        mh = m / (1 - beta1 ** t)
        vh = v / (1 - beta2 ** t)
        out[k] = np.asarray(params[k], np.float64) - lr * mh / (np.sqrt(vh) + eps)
    return out
