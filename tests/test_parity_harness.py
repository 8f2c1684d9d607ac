"""CPU checks of the GPU parity harness (tests/parity.py): the oracle's own
rollout stands in for the device's, and mistakes are planted in that copy.

* an identical copy shows no divergence;
* a flipped action, a latent drawn from another component and a flipped
  done flag, each away from a near-tie, are rejected;
* a flip that the recorded state drift explains (the copy's state moved,
  and its action is the one the moved state picks) is accepted and counted;
* the near-tie cap has no floor.
"""

import copy
import sys

import numpy as np
import pytest

import parity
from oracle import philox as ph
from oracle import wm as owm
from paper_2205_01435_amd import workloads as wl

SEED = 7


@pytest.fixture(scope="module")
def case():
    w = wl.Workload("h", "rollout", B=6, T=5, Z=8, H=16, A=5, K=3, dtype="fp32", seed=3, mask_p=0.8)
    inp = wl.make_rollout_inputs(w)
    ref = owm.rollout(inp["weights"], w.dims, inp["z0"], inp["mask"], T=w.T, seed=SEED, tau=1.0,
                      done_flag=True)
    return w, inp, ref


def _run(w, inp, ref, g):
    return parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=inp["mask"], seed=SEED)


def _live_step(ref, b_min=0):
    """(b, t) of a live step with at least two valid actions."""
    for b in range(b_min, ref["actions"].shape[1]):
        for t in range(ref["actions"].shape[0]):
            if ref["actions"][t, b] >= 0 and np.isfinite(ref["action_margin"][t, b]):
                return b, t
    raise AssertionError("no live step")


def test_identical_copy_has_no_divergence(case):
    w, inp, ref = case
    rec = {}
    assert parity.free_run(ref, copy.deepcopy(ref), weights=inp["weights"], dims=w.dims,
                           mask=inp["mask"], seed=SEED, record=rec) == 0
    assert rec["free_run_diverged"] == 0 and rec["free_run_steps_compared"] > 0


def test_flipped_action_away_from_a_tie_is_rejected(case):
    w, inp, ref = case
    b, t = _live_step(ref)
    assert ref["action_margin"][t, b] > 1e-3
    g = copy.deepcopy(ref)
    valid = np.nonzero(inp["mask"][b])[0]
    g["actions"][t, b] = valid[valid != ref["actions"][t, b]][0]
    with pytest.raises(AssertionError, match="without a near-tie"):
        _run(w, inp, ref, g)


def test_other_component_draw_is_rejected(case):
    w, inp, ref = case
    b, t = _live_step(ref)
    wb = owm.weight_blocks(inp["weights"], w.Z, w.H, w.A, w.K, "fp32")
    h1 = ref["h_trace"][t + 1, b][None]
    pi, mu, ls = owm.mdn_params(wb, h1, w.Z, w.K, "fp32")
    u1 = ph.stream_uniforms(SEED, np.array([b]), t, ph.STREAM_COMPONENT, w.Z * w.K).reshape(w.Z, w.K)
    eps = owm.box_muller(ph.stream_uniforms(SEED, np.array([b]), t, ph.STREAM_GAUSS, w.Z))[0]
    sc = pi[0] + owm.gumbel(u1)
    order = np.argsort(sc, axis=-1)
    gaps = sc[np.arange(w.Z), order[:, -1]] - sc[np.arange(w.Z), order[:, -2]]
    j = int(np.argmax(gaps))  # the dim farthest from a tie
    k2 = order[j, -2]
    g = copy.deepcopy(ref)
    g["z_out"][t + 1, b, j] = mu[0, j, k2] + np.exp(ls[0, j, k2]) * eps[j]
    with pytest.raises(AssertionError, match="without a near-tie"):
        _run(w, inp, ref, g)


def test_flipped_done_away_from_a_tie_is_rejected(case):
    w, inp, ref = case
    live = np.argwhere((ref["actions"] >= 0) & (ref["done_margin"] > 1e-2))
    t, b = live[0]
    g = copy.deepcopy(ref)
    g["dones"][t, b] = 1 - g["dones"][t, b]
    with pytest.raises(AssertionError, match="done flips"):
        _run(w, inp, ref, g)


def test_flip_explained_by_state_drift_is_accepted(case, monkeypatch):
    """The copy's h_t moves (the float bar is opened for this test) and its
    action is the one the moved state picks: the drift term explains it."""
    w, inp, ref = case
    monkeypatch.setitem(parity.RTOL, "fp32", 1e6)
    b, t = _live_step(ref)
    wb = owm.weight_blocks(inp["weights"], w.Z, w.H, w.A, w.K, "fp32")
    u0 = ph.stream_uniforms(SEED, np.array([b]), t, ph.STREAM_CONTROLLER, w.A)[0]
    z, h = ref["z_out"][t, b], ref["h_trace"][t, b]
    ar = ref["actions"][t, b]
    valid = np.nonzero(inp["mask"][b])[0]
    alt = valid[valid != ar][0]
    # move h along the controller rows' difference until `alt` wins
    d = wb["W_c"][alt, w.Z:] - wb["W_c"][ar, w.Z:]
    s0 = owm.controller_logits(wb, z[None], h[None], "fp32")[0] + owm.gumbel(u0)
    gap = s0[ar] - s0[alt]
    h2 = h + d * (1.5 * gap / np.dot(d, d))
    s2 = owm.controller_logits(wb, z[None], h2[None], "fp32")[0] + owm.gumbel(u0)
    assert s2[alt] > s2[ar]
    g = copy.deepcopy(ref)
    g["h_trace"][t, b] = h2
    g["actions"][t, b] = int(np.argmax(np.where(inp["mask"][b] != 0, s2, -np.inf)))
    rec = {}
    assert parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=inp["mask"], seed=SEED,
                           record=rec) == 1
    assert rec["free_run_kinds"]["action"] == 1
    # the same flip without the drift is rejected
    g["h_trace"][t, b] = h
    with pytest.raises(AssertionError, match="without a near-tie"):
        _run(w, inp, ref, g)


def test_caps():
    c = parity.TieCounter()
    c.draws, c.mismatches = 999, 1
    with pytest.raises(AssertionError):
        c.check()  # 1 of 999 draws is above 0.1 %: no floor of one mismatch
    c.draws = 1000
    c.check()
    assert parity.free_run_cap(16) == 1 and parity.free_run_cap(5000) == 5


if __name__ == "__main__":
    sys.exit(pytest.main([__file__, "-q"]))
