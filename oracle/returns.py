"""Float64 oracle of the return scan over dreamed trajectories.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The agent looks for the policy that maximises the expected discounted sum of
rewards, with a discount factor gamma in [0, 1) (section 2.2, the
reinforcement-learning objective).  Its controller is trained with PPO
(sections 2.3 and 4.1), and a PPO update on dreamed
trajectories needs, for every trajectory and step, the discounted return
and, given a value baseline, the generalised advantage estimate (GAE(lambda),
Schulman et al., ICLR 2016).

Readings (also listed in the design notes):
* a step with done_t = 1 ends its trajectory: nothing after it is discounted
  into step t.  The frozen steps a rollout emits after a done (reward 0,
  done 1) therefore add nothing.
* without values, the return after the last step is 0 (no bootstrap):
      G_t = r_t + gamma (1 - d_t) G_{t+1},   G_T = 0;
* with values V [T+1, B] (V_T bootstraps the tail):
      delta_t = r_t + gamma (1 - d_t) V_{t+1} - V_t
      A_t     = delta_t + gamma lambda (1 - d_t) A_{t+1},   A_T = 0
      ret_t   = A_t + V_t
  (lambda = 1 gives the discounted return bootstrapped by V_T).
"""

from __future__ import annotations

import numpy as np


def returns(rewards, dones, gamma: float, values=None, lam: float = 1.0):
    """(returns [T, B], advantages [T, B] or None), float64, by the backward
    recursions above, one step at a time."""
    r = np.asarray(rewards, np.float64)
    d = np.asarray(dones).astype(np.float64)
    T = r.shape[0]
    cont = 1.0 - d  # 0 where the trajectory ends at this step
    if values is None:
        G = np.zeros_like(r)
        nxt = np.zeros(r.shape[1:], np.float64)
        for t in range(T - 1, -1, -1):
            nxt = r[t] + gamma * cont[t] * nxt
            G[t] = nxt
        return G, None
    V = np.asarray(values, np.float64)
    assert V.shape[0] == T + 1
    A = np.zeros_like(r)
    nxt = np.zeros(r.shape[1:], np.float64)
    for t in range(T - 1, -1, -1):
        delta = r[t] + gamma * cont[t] * V[t + 1] - V[t]
        nxt = delta + gamma * lam * cont[t] * nxt
        A[t] = nxt
    return A + V[:T], A
