"""Seeded synthetic workloads for the World-Model dream rollout and NLL pass.

This module only draws input data (weights, latents, masks, logged
sequences) from a seeded numpy generator.  It holds none of the model's
arithmetic, and both the CPU oracle tests and the HIP path consume the
arrays it returns.

Shapes follow the paper's World Model (RLFlow, section 3.3, "World Models"):
a recurrent mixture-density model over a latent ``z`` of size ``Z`` with an
LSTM hidden state of size ``H``, ``A`` discrete graph-transformation actions
and ``K`` Gaussians per latent dimension.  The paper reports 8 Gaussians and
256 hidden units (section 4.7) and action spaces of order 10^2 (Table 1);
the five workloads below stretch those to the sizes used for measurement.

Draw order (fixed; a change here changes every workload):
  1. weights, in the order W_g, W_m, w_r, w_d, W_c, each Xavier-uniform on
     its canonical ``[out, in]`` shape, drawn in float64 and stored float32;
  2. rollout: ``z0 ~ N(0, 1)`` of shape ``[B, Z]``;
     NLL: the logged sequences (see ``make_nll_inputs``);
  3. the valid-action mask: ``U ~ U[0,1)^{B x A}``, ``mask = U < p``; a row
     left empty gets ``mask[b, argmin_a U[b, a]] = 1``.
Biases are zero except the done head's, which is ``logit(1/T)`` so that a
trajectory stops with probability about ``1/T`` per step.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = [
    "Workload",
    "WORKLOADS",
    "xavier_uniform",
    "make_weights",
    "make_mask",
    "make_rollout_inputs",
    "make_nll_inputs",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload: model dims, batch, horizon and generators."""

    name: str
    kind: str  # "rollout" or "nll"
    B: int
    T: int
    Z: int
    H: int
    A: int
    K: int
    dtype: str  # "fp32" or "bf16" (weights and activations; fp32 accumulate)
    seed: int
    mask_p: float = 0.3
    done: bool = True  # done head active in rollouts
    tau: float = 1.0
    ar_rho: float = 0.9  # NLL latents: AR(1) coefficient
    reward_std: float = 0.1  # NLL logged rewards

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def dims(self) -> dict:
        return dict(Z=self.Z, H=self.H, A=self.A, K=self.K)


# The five measured workloads, smallest first.
WORKLOADS = {
    "tiny_rollout": Workload("tiny_rollout", "rollout", B=16, T=20, Z=32, H=256, A=32, K=5,
                             dtype="fp32", seed=0, mask_p=0.3, done=False),
    "medium_rollout": Workload("medium_rollout", "rollout", B=256, T=50, Z=64, H=512, A=64, K=5,
                               dtype="fp32", seed=1, mask_p=0.3, done=True),
    "nll": Workload("nll", "nll", B=512, T=128, Z=64, H=512, A=64, K=5,
                    dtype="fp32", seed=2, mask_p=0.3),
    "large_rollout": Workload("large_rollout", "rollout", B=4096, T=100, Z=64, H=1024, A=128, K=8,
                              dtype="bf16", seed=3, mask_p=0.3, done=True),
    "xlarge_rollout": Workload("xlarge_rollout", "rollout", B=16384, T=64, Z=128, H=1024, A=256,
                               K=8, dtype="bf16", seed=4, mask_p=0.1, done=True),
}


def xavier_uniform(rng: np.random.Generator, out_features: int, in_features: int) -> np.ndarray:
    """Glorot/Xavier uniform U(-a, a), a = sqrt(6 / (fan_in + fan_out)), float32."""
    a = math.sqrt(6.0 / (in_features + out_features))
    return rng.uniform(-a, a, size=(out_features, in_features)).astype(np.float32)


def make_weights(rng: np.random.Generator, Z: int, H: int, A: int, K: int, T: int) -> dict:
    """Canonical float32 weights.

    Layouts (row-major ``[out, in]``):
      W_g [4H, Z+A+H]  rows gate-major (i | f | g | o), columns z | one-hot a | h
      W_m [3ZK, H]     row p*Z*K + j*K + k, p = 0 logit-pi, 1 mu, 2 log-sigma
      w_r [H], w_d [H] reward and done heads on h_{t+1}
      W_c [A, Z+H]     controller, columns z | h
    """
    W_g = xavier_uniform(rng, 4 * H, Z + A + H)
    W_m = xavier_uniform(rng, 3 * Z * K, H)
    w_r = xavier_uniform(rng, 1, H)[0]
    w_d = xavier_uniform(rng, 1, H)[0]
    W_c = xavier_uniform(rng, A, Z + H)
    p_done = 1.0 / max(T, 1)
    b_d = math.log(p_done / (1.0 - p_done)) if p_done < 1.0 else 30.0
    return dict(
        W_g=W_g, b_g=np.zeros(4 * H, np.float32),
        W_m=W_m, b_m=np.zeros(3 * Z * K, np.float32),
        w_r=w_r, b_r=np.float32(0.0),
        w_d=w_d, b_d=np.float32(b_d),
        W_c=W_c, b_c=np.zeros(A, np.float32),
    )


def make_mask(rng: np.random.Generator, B: int, A: int, p: float) -> np.ndarray:
    """Bernoulli(p) valid-action mask ``[B, A]`` (uint8) with >= 1 valid per row."""
    U = rng.random((B, A))
    mask = (U < p).astype(np.uint8)
    empty = mask.sum(axis=1) == 0
    if empty.any():
        rows = np.nonzero(empty)[0]
        mask[rows, np.argmin(U[rows], axis=1)] = 1
    return mask


def make_rollout_inputs(w: Workload, B: int | None = None) -> dict:
    """Inputs of a dream rollout: weights, ``z0 [B, Z]``, ``mask [B, A]``.

    ``h0 = c0 = 0`` (not stored).  ``B`` may override the workload's batch
    size; the draws then differ, which is harmless because every consumer
    receives the same arrays.
    """
    B = w.B if B is None else B
    rng = np.random.Generator(np.random.PCG64(w.seed))
    weights = make_weights(rng, w.Z, w.H, w.A, w.K, w.T)
    z0 = rng.standard_normal((B, w.Z)).astype(np.float32)
    mask = make_mask(rng, B, w.A, w.mask_p)
    return dict(weights=weights, z0=z0, mask=mask)


def make_nll_inputs(w: Workload, B: int | None = None, T: int | None = None) -> dict:
    """Logged sequences for the teacher-forced NLL pass.

    Draw order after the weights:
      latents ``z [T+1, B, Z]``: ``e ~ N(0,1)``, ``z_0 = e_0``,
        ``z_t = rho z_{t-1} + sqrt(1 - rho^2) e_t`` (stationary N(0,1) AR(1));
      mask ``[B, A]`` as for rollouts;
      actions ``[T, B]``: ``idx = floor(U * nvalid[b])``, the idx-th valid action
        of row b (uniform over the valid set, the random agent of section 3.3.2);
      rewards ``[T, B]`` ``~ N(0, reward_std^2)``;
      dones ``[T, B]`` ``~ Bernoulli(1/T)``.
    """
    B = w.B if B is None else B
    T = w.T if T is None else T
    rng = np.random.Generator(np.random.PCG64(w.seed))
    weights = make_weights(rng, w.Z, w.H, w.A, w.K, T)
    e = rng.standard_normal((T + 1, B, w.Z))
    z = np.empty_like(e)
    z[0] = e[0]
    s = math.sqrt(1.0 - w.ar_rho ** 2)
    for t in range(1, T + 1):
        z[t] = w.ar_rho * z[t - 1] + s * e[t]
    mask = make_mask(rng, B, w.A, w.mask_p)
    nvalid = mask.sum(axis=1).astype(np.int64)
    idx = np.floor(rng.random((T, B)) * nvalid[None, :]).astype(np.int64)
    idx = np.minimum(idx, nvalid[None, :] - 1)
    valid_lists = [np.nonzero(mask[b])[0] for b in range(B)]
    actions = np.empty((T, B), np.int32)
    for b in range(B):
        actions[:, b] = valid_lists[b][idx[:, b]]
    rewards = (w.reward_std * rng.standard_normal((T, B))).astype(np.float32)
    dones = (rng.random((T, B)) < 1.0 / max(T, 1)).astype(np.uint8)
    return dict(weights=weights, z=z.astype(np.float32), actions=actions,
                rewards=rewards, dones=dones, mask=mask)
