"""Parity helpers: compare the HIP path (through the C ABI) with the oracle.

Rules (fixed here, used by every GPU test):
* Floats: ``|gpu - ref| <= rtol * (|ref| + rms(ref))`` per tensor and step,
  rtol = 1e-4 for fp32 workloads and 2e-2 for bf16 ones.
* Discrete outputs (actions, mixture components, done flags) must be equal,
  except at near-ties: the oracle's float64 gap between the two best Gumbel
  scores (or |sigmoid(rho_d) - u| for done) below ``eps * (1 + |s1|)``.
  Every mismatch must be a near-tie, and mismatches are capped at 0.1 % of
  the draws compared.
* Re-anchored mode: for every step the oracle restarts from the device's own
  state (z_t, h_t, c_t, done flags from its trace) and recomputes one step,
  with the mixture head fed the device's h_{t+1}; errors cannot compound.
* Free-run mode: whole trajectories are compared up to their first
  divergence, which must start at a near-tie, with the bound widened by the
  exact score change the two runs' accumulated state drift causes; diverged
  trajectories are capped at 0.1 % of the batch (at least one).
* Near-tie counts of every comparison can be appended to a JSON-lines file
  named by the environment variable WM_TIE_RECORD (``record_ties``).
"""

from __future__ import annotations

import json
import os

import numpy as np
from scipy.special import expit

from oracle import wm as owm

RTOL = {"fp32": 1e-4, "bf16": 2e-2}
EPS_TIE = {"fp32": 1e-5, "bf16": 1e-3}
TIE_CAP = 1e-3


def record_ties(case: str, **counts):
    """Append one JSON line of near-tie counts for ``case`` to $WM_TIE_RECORD."""
    path = os.environ.get("WM_TIE_RECORD")
    if not path:
        return
    with open(path, "a") as f:
        f.write(json.dumps({"case": case, **{k: (v if not isinstance(v, np.generic) else v.item())
                                              for k, v in counts.items()}}) + "\n")


def close(gpu, ref, rtol, what=""):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    if ref.size == 0:
        return
    scale = np.sqrt(np.mean(ref ** 2))
    err = np.abs(gpu - ref)
    tol = rtol * (np.abs(ref) + scale) + 1e-30
    bad = err > tol
    if bad.any():
        i = np.unravel_index(np.argmax(err / tol), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} beyond rtol={rtol}; worst at {i}: "
                             f"gpu={gpu[i]!r} ref={ref[i]!r}")


def elem_close(gpu, ref, rtol, scale):
    return np.abs(np.asarray(gpu, np.float64) - ref) <= rtol * (np.abs(ref) + scale)


class TieCounter:
    def __init__(self):
        self.draws = 0
        self.mismatches = 0

    def check(self, cap=TIE_CAP):
        assert self.mismatches <= cap * self.draws, \
            f"{self.mismatches} near-tie mismatches in {self.draws} draws exceed {cap:.1%}"


def check_padding(g, t, rows):
    """Rows past their horizon at step t show the padding pattern: action -1,
    reward 0, done 0, zero latent, state unchanged."""
    if rows.size == 0:
        return
    assert np.all(g["actions"][t][rows] == -1) and np.all(g["rewards"][t][rows] == 0)
    assert np.all(g["dones"][t][rows] == 0)
    assert np.all(g["z_out"][t + 1][rows] == 0)
    if "h_trace" in g:
        np.testing.assert_array_equal(g["h_trace"][t + 1][rows], g["h_trace"][t][rows])
        np.testing.assert_array_equal(g["c_trace"][t + 1][rows], g["c_trace"][t][rows])


def reanchored(dims, wts, mask, g, *, seed, tau, done_flag, dtype, traj=None, step0=0,
               done0=None, sigma_tau=False, two_level=None, lengths=None):
    """Re-anchored comparison of a device rollout.

    ``g`` holds the device's z_out, actions, rewards, dones, h_trace and
    c_trace for some trajectories (batch axis of length n), ``mask [n, A]``
    (or [T, n, A] per step) their masks and ``traj [n]`` their trajectory indices (default 0..n-1).
    ``lengths [n]``: per-trajectory horizons; later steps must be padding.
    """
    T = g["actions"].shape[0]
    n = g["actions"].shape[1]
    traj = np.arange(n) if traj is None else np.asarray(traj)
    rtol, eps = RTOL[dtype], EPS_TIE[dtype]
    wb = owm.weight_blocks(wts, dims["Z"], dims["H"], dims["A"], dims["K"], dtype)
    ties = TieCounter()
    live = np.ones(n, bool) if done0 is None else np.asarray(done0) == 0
    n_live_steps = 0
    horizon = np.full(n, T) if lengths is None else np.asarray(lengths)
    for t in range(T):
        za, ha, ca = g["z_out"][t], g["h_trace"][t], g["c_trace"][t]
        a_g = g["actions"][t]
        inside = t < horizon
        check_padding(g, t, np.nonzero(~inside)[0])
        # frozen rows must show the frozen pattern
        fr = ~live & inside
        assert np.all(a_g[fr] == -1) and np.all(g["dones"][t][fr] == 1)
        assert np.all(g["rewards"][t][fr] == 0)
        np.testing.assert_array_equal(g["z_out"][t + 1][fr], za[fr])
        idx = np.nonzero(live & inside)[0]
        if idx.size == 0:
            continue
        n_live_steps += idx.size
        sel = idx
        if two_level is not None:  # (xfer masks, location masks)
            m_sel = (mask[0][sel], mask[1][sel])
        else:
            mask_t = mask[t] if mask.ndim == 3 else mask  # per-step masks: [T, n, A]
            m_sel = mask_t[sel]
        r = owm.transition(wb, dims, za[idx], ha[idx], ca[idx], m_sel, seed=seed,
                           traj=traj[sel], step=step0 + t, tau=tau, done_flag=done_flag,
                           dtype=dtype, h_next=g["h_trace"][t + 1][sel], sigma_tau=sigma_tau,
                           two_level=two_level)
        # actions
        ag = a_g[idx]
        ties.draws += idx.size
        diff = ag != r["action"]
        if diff.any():
            near = r["action_margin"][diff] < eps * (1 + np.abs(r["action_top"][diff]))
            assert near.all(), (f"step {t}: action mismatch at non-tie rows {sel[diff][~near]}, "
                                f"gpu={ag[diff][~near]} ref={r['action'][diff][~near]}, "
                                f"margin={r['action_margin'][diff][~near]}")
            ties.mismatches += int(diff.sum())
            r2 = owm.transition(wb, dims, za[idx], ha[idx], ca[idx], m_sel, seed=seed,
                                traj=traj[sel], step=step0 + t, tau=tau, done_flag=done_flag,
                                dtype=dtype, h_next=g["h_trace"][t + 1][sel], action=ag,
                                sigma_tau=sigma_tau, two_level=two_level)
            r["h"], r["c"] = r2["h"], r2["c"]
        ok = ag >= 0
        # state
        close(g["h_trace"][t + 1][sel][ok], r["h"][ok], rtol, f"h step {t}")
        close(g["c_trace"][t + 1][sel][ok], r["c"][ok], rtol, f"c step {t}")
        # latent draw: per (row, dim) agreement or a component near-tie
        zg = g["z_out"][t + 1][sel][ok]
        zr = r["z"][ok]
        scale = np.sqrt(np.mean(zr ** 2)) if zr.size else 0.0
        good = elem_close(zg, zr, rtol, scale)
        ties.draws += zg.size
        if not good.all():
            km = r["component_margin"][ok][~good]
            kt = r["component_top"][ok][~good]
            near = km < eps * (1 + np.abs(kt))
            assert near.all(), f"step {t}: z mismatch without a component near-tie ({(~near).sum()})"
            ties.mismatches += int((~good).sum())
        close(g["rewards"][t][sel][ok], r["reward"][ok], rtol, f"reward step {t}")
        dg = g["dones"][t][sel][ok].astype(bool)
        dr = r["done"][ok]
        ties.draws += dg.size
        dd = dg != dr
        if dd.any():
            u3m = r["done_margin"][ok][dd]
            assert np.all(u3m < eps), f"step {t}: done mismatch away from a tie: {u3m}"
            ties.mismatches += int(dd.sum())
        # rows without a valid action end with the frozen pattern
        na = ~ok
        if na.any():
            assert np.all(g["dones"][t][sel][na] == 1) and np.all(g["rewards"][t][sel][na] == 0)
        done_now = np.zeros(idx.size, bool)
        done_now[ok] = dg
        new_live = live.copy()
        new_live[idx] = ok & ~done_now
        live = new_live
    ties.check()
    return ties, n_live_steps


def free_run_cap(B: int) -> float:
    """Largest number of diverged trajectories a free-run comparison of B
    trajectories may show: 0.1 % of them, and at least one."""
    return max(1.0, TIE_CAP * B)


def free_run(ref, g, *, weights, dims, mask, seed, tau=1.0, dtype="fp32", traj=None, step0=0,
             sigma_tau=False, record=None, lengths=None):
    """Free-run comparison of a device rollout ``g`` with the oracle's own
    rollout ``ref`` of the same inputs.

    Each trajectory is followed step by step while the two agree: the state
    entering the step (z_t, and h_t when the device trace is there) within
    the float bar, the same action, every latent dim of z_{t+1} within the
    float bar, the same done flag and the reward within the float bar.  The
    first step where a discrete decision differs ends the comparison of that
    trajectory (it has diverged) and must be explained by a near-tie:

      the oracle's own score gap between its pick and the device's pick is
      at most  eps (1 + |s1|) + |d(pick_ref) - d(pick_dev)|,

    where eps is the re-anchored near-tie bound of the dtype and d is the
    exact (float64) change of the two competing scores caused by the state
    drift the two runs have accumulated so far: the scores recomputed from
    the device's own state minus the oracle's (the random streams are the
    same on both sides, so they cancel).  For the done flag the bound is on
    |sigmoid(rho_d) - u|.  The device's mixture component is identified from
    its z_{t+1}: the component whose draw from the device's own h_{t+1}
    reproduces it.  Float disagreement without a discrete flip fails.

    Returns the number of diverged trajectories; ``record`` (a dict) gets the
    counts.  Without a device trace the drift term is 0 (the bound is the
    re-anchored one).  With ``lengths`` the steps past a trajectory's horizon
    must be padding on both sides.
    """
    from oracle import philox as ph

    rtol, eps = RTOL[dtype], EPS_TIE[dtype]
    Z, H, A, K = dims["Z"], dims["H"], dims["A"], dims["K"]
    T = g["actions"].shape[0]
    B = g["actions"].shape[1]
    traj = np.arange(B) if traj is None else np.asarray(traj)
    wb = owm.weight_blocks(weights, Z, H, A, K, dtype)
    mask = np.asarray(mask)
    has_h = "h_trace" in g
    zs = np.sqrt(np.mean(ref["z_out"] ** 2))
    hs = np.sqrt(np.mean(ref["h_trace"] ** 2))
    rs = np.sqrt(np.mean(ref["rewards"] ** 2)) + 1e-30
    sig = np.sqrt(tau) if sigma_tau else 1.0
    diverged, compared, worst = 0, 0, 0.0
    kinds = {"action": 0, "component": 0, "done": 0}
    for b in range(B):
        tb = traj[b:b + 1]
        for t in range(T):
            s = step0 + t
            if lengths is not None and t >= lengths[b]:
                check_padding(g, t, np.array([b]))
                check_padding(ref, t, np.array([b]))
                continue
            zr, hr = ref["z_out"][t, b], ref["h_trace"][t, b]
            zg = g["z_out"][t, b]
            hg = g["h_trace"][t, b] if has_h else hr
            assert np.all(elem_close(zg, zr, rtol, zs)), f"traj {b} step {t}: z_t drifted beyond rtol"
            assert np.all(elem_close(hg, hr, rtol, hs)), f"traj {b} step {t}: h_t drifted beyond rtol"
            ar, ag = int(ref["actions"][t, b]), int(g["actions"][t, b])
            frozen = ar < 0 and ag < 0
            if frozen:
                assert g["dones"][t, b] == 1 and g["rewards"][t, b] == 0
                continue
            compared += 1
            m_t = mask[t] if mask.ndim == 3 else mask
            if ar != ag:
                # controller scores from both states; the Gumbel noise is shared
                u0 = ph.stream_uniforms(seed, tb, s, ph.STREAM_CONTROLLER, A)[0]
                lr = owm.controller_logits(wb, zr[None], hr[None], dtype)[0]
                lg = owm.controller_logits(wb, zg[None], hg[None], dtype)[0]
                assert ar >= 0 and ag >= 0 and m_t[b, ag], \
                    f"traj {b} step {t}: action {ag} vs {ar} (invalid or missing pick)"
                sr = lr + owm.gumbel(u0)
                gap = sr[ar] - sr[ag]
                drift = abs((lg[ar] - lr[ar]) - (lg[ag] - lr[ag]))
                bound = eps * (1 + abs(sr[ar])) + drift
                assert gap <= bound, (f"traj {b} diverges at step {t} without a near-tie: action {ag} vs "
                                      f"{ar}, oracle gap {gap:.3g} > bound {bound:.3g} (drift {drift:.3g})")
                diverged += 1
                kinds["action"] += 1
                worst = max(worst, gap)
                break
            # the step's state, rewards and latent draw
            hr1 = ref["h_trace"][t + 1, b]
            hg1 = g["h_trace"][t + 1, b] if has_h else hr1
            assert np.all(elem_close(hg1, hr1, rtol, hs)), f"traj {b} step {t}: h_t+1 beyond rtol"
            zr1, zg1 = ref["z_out"][t + 1, b], g["z_out"][t + 1, b]
            zok = elem_close(zg1, zr1, rtol, zs)
            if not zok.all():
                pr, mur, lsr = owm.mdn_params(wb, hr1[None], Z, K, dtype)
                pg, mug, lsg = owm.mdn_params(wb, hg1[None], Z, K, dtype)
                u1 = ph.stream_uniforms(seed, tb, s, ph.STREAM_COMPONENT, Z * K).reshape(Z, K)
                u2 = ph.stream_uniforms(seed, tb, s, ph.STREAM_GAUSS, Z)
                e = owm.box_muller(u2)[0]
                sr = pr[0] / tau + owm.gumbel(u1)
                for j in np.nonzero(~zok)[0]:
                    kr = int(np.argmax(sr[j]))
                    cand = mug[0, j] + np.exp(lsg[0, j]) * sig * e[j]  # device draw per component
                    kg = int(np.argmin(np.abs(cand - zg1[j])))
                    assert kg != kr and elem_close(zg1[j], cand[kg], rtol, zs), \
                        (f"traj {b} step {t} dim {j}: z {zg1[j]!r} vs {zr1[j]!r} matches no other "
                         f"component's draw")
                    gap = sr[j, kr] - sr[j, kg]
                    drift = abs(((pg[0, j, kr] - pr[0, j, kr]) - (pg[0, j, kg] - pr[0, j, kg])) / tau)
                    bound = eps * (1 + abs(sr[j, kr])) + drift
                    assert gap <= bound, (f"traj {b} diverges at step {t} dim {j} without a near-tie: "
                                          f"component {kg} vs {kr}, gap {gap:.3g} > bound {bound:.3g}")
                    worst = max(worst, gap)
                diverged += 1
                kinds["component"] += 1
                break
            assert abs(g["rewards"][t, b] - ref["rewards"][t, b]) <= \
                rtol * (abs(ref["rewards"][t, b]) + rs), f"traj {b} step {t}: reward beyond rtol"
            if g["dones"][t, b] != ref["dones"][t, b]:
                u3 = ph.stream_uniforms(seed, tb, s, ph.STREAM_DONE, 1)[0, 0]
                _, rdr = owm.reward_done_logits(wb, hr1[None], dtype)
                _, rdg = owm.reward_done_logits(wb, hg1[None], dtype)
                pr_, pg_ = float(expit(rdr[0])), float(expit(rdg[0]))
                gap = abs(pr_ - u3)
                bound = eps + abs(pg_ - pr_)
                assert gap <= bound, (f"traj {b} done flips at step {t} without a near-tie: "
                                      f"|p - u| = {gap:.3g} > {bound:.3g}")
                diverged += 1
                kinds["done"] += 1
                worst = max(worst, gap)
                break
    if record is not None:
        record.update(free_run_rows=B, free_run_diverged=diverged, free_run_steps_compared=compared,
                      free_run_kinds=kinds, free_run_worst_gap=worst)
    return diverged
