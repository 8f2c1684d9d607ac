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
  divergence, which must start at a near-tie.
"""

from __future__ import annotations

import numpy as np

from oracle import wm as owm

RTOL = {"fp32": 1e-4, "bf16": 2e-2}
EPS_TIE = {"fp32": 1e-5, "bf16": 1e-3}
# free-run: an absolute margin, wider because the state error compounds over steps
EPS_TIE_FREE = {"fp32": 1e-3, "bf16": 1e-2}
TIE_CAP = 1e-3


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
        assert self.mismatches <= max(1, cap * self.draws), \
            f"{self.mismatches} near-tie mismatches in {self.draws} draws exceed {cap:.1%}"


def reanchored(dims, wts, mask, g, *, seed, tau, done_flag, dtype, traj=None, step0=0,
               done0=None, sigma_tau=False, two_level=None):
    """Re-anchored comparison of a device rollout.

    ``g`` holds the device's z_out, actions, rewards, dones, h_trace and
    c_trace for some trajectories (batch axis of length n), ``mask [n, A]``
    (or [T, n, A] per step) their masks and ``traj [n]`` their trajectory indices (default 0..n-1).
    """
    T = g["actions"].shape[0]
    n = g["actions"].shape[1]
    traj = np.arange(n) if traj is None else np.asarray(traj)
    rtol, eps = RTOL[dtype], EPS_TIE[dtype]
    wb = owm.weight_blocks(wts, dims["Z"], dims["H"], dims["A"], dims["K"], dtype)
    ties = TieCounter()
    live = np.ones(n, bool) if done0 is None else np.asarray(done0) == 0
    n_live_steps = 0
    for t in range(T):
        za, ha, ca = g["z_out"][t], g["h_trace"][t], g["c_trace"][t]
        a_g = g["actions"][t]
        # frozen rows must show the frozen pattern
        fr = ~live
        assert np.all(a_g[fr] == -1) and np.all(g["dones"][t][fr] == 1)
        assert np.all(g["rewards"][t][fr] == 0)
        np.testing.assert_array_equal(g["z_out"][t + 1][fr], za[fr])
        idx = np.nonzero(live)[0]
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


def free_run(ref, g, dtype, T):
    """Free-run comparison: per trajectory, equal up to the first divergence,
    which must follow a near-tie; returns the number of diverged rows."""
    rtol = RTOL[dtype]
    eps = EPS_TIE_FREE[dtype]
    B = g["actions"].shape[1]
    zs = np.sqrt(np.mean(ref["z_out"] ** 2))
    rs = np.sqrt(np.mean(ref["rewards"] ** 2)) + 1e-30
    diverged = 0
    for b in range(B):
        for t in range(T):
            a_ok = g["actions"][t, b] == ref["actions"][t, b]
            d_ok = g["dones"][t, b] == ref["dones"][t, b]
            zok = elem_close(g["z_out"][t + 1, b], ref["z_out"][t + 1, b], rtol, zs)
            r_ok = abs(g["rewards"][t, b] - ref["rewards"][t, b]) <= rtol * (abs(ref["rewards"][t, b]) + rs)
            if a_ok and d_ok and zok.all() and r_ok:
                continue
            # first divergence: it must sit at a near-tie of this step
            am = ref["action_margin"][t, b]
            km = ref["component_margin"][t, b]
            dm = ref["done_margin"][t, b]
            tie = (not a_ok and am < eps) or \
                  (a_ok and not zok.all() and np.all(km[~zok] < eps)) or \
                  (a_ok and zok.all() and not d_ok and dm < eps)
            assert tie, (f"traj {b} diverges at step {t} without a near-tie: actions "
                         f"{g['actions'][t, b]} vs {ref['actions'][t, b]} (margin {am}), "
                         f"dones {g['dones'][t, b]} vs {ref['dones'][t, b]} (margin {dm}), "
                         f"z ok {zok.sum()}/{zok.size}, reward {g['rewards'][t, b]} vs "
                         f"{ref['rewards'][t, b]}")
            diverged += 1
            break
    return diverged
