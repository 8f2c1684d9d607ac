"""GPU parity of the HIP path (called through the C ABI) against the oracle.

Run on an MI355X: ``python -m pytest tests -m gpu``.  Inputs are the seeded
synthetic workloads of ``paper_2205_01435_amd.workloads``; both sides consume
the same arrays and the same Philox streams.
"""

import sys

import numpy as np
import pytest
import torch

import parity
from oracle import wm as owm
from paper_2205_01435_amd import _lib as wmlib
from paper_2205_01435_amd import workloads as wl

pytestmark = pytest.mark.gpu

ROLL_KEYS = ("z_out", "actions", "rewards", "dones", "h_T", "c_T", "h_trace", "c_trace")


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    wmlib.load()
    yield


def _t(x, dtype=None):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda() if dtype is None else \
        torch.from_numpy(np.ascontiguousarray(x)).to(dtype).cuda()


def run_rollout(w, inp, *, T=None, trace=True, seed=None, tau=None, done=None, traj0=0,
                step0=0, h0=None, c0=None, done_io=None, model=None, rows=None):
    T = w.T if T is None else T
    m = model or wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0 = inp["z0"] if rows is None else inp["z0"][rows]
    mask = inp["mask"] if rows is None else inp["mask"][rows]
    dio = None if done_io is None else _t(done_io)
    b = wmlib.rollout(m, _t(z0), _t(mask), T=T, seed=w.seed if seed is None else seed,
                      tau=w.tau if tau is None else tau, done=w.done if done is None else done,
                      traj0=traj0, step0=step0, h0=None if h0 is None else _t(h0),
                      c0=None if c0 is None else _t(c0), done_io=dio, trace=trace)
    torch.cuda.synchronize()
    out = {k: getattr(b, k).cpu().numpy() for k in ROLL_KEYS if getattr(b, k) is not None}
    if dio is not None:
        out["done_io"] = dio.cpu().numpy()
    return out


# ---------------------------------------------------------------------------
# controller step
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,B,Z,H,A", [("fp32", 37, 64, 512, 64), ("bf16", 100, 128, 1024, 256),
                                           ("fp32", 19, 8, 48, 37),
                                           # wide controllers (more than 318 logit rows): 8, 24
                                           # and 33 output blocks per wave
                                           ("fp32", 37, 64, 512, 500), ("fp32", 21, 16, 64, 1100),
                                           ("bf16", 70, 64, 256, 2000)])
def test_controller_step(dtype, B, Z, H, A):
    say("controller_step", dtype, B, Z, H, A)
    w = wl.Workload("c", "rollout", B=B, T=10, Z=Z, H=H, A=A, K=2, dtype=dtype, seed=21)
    inp = wl.make_rollout_inputs(w)
    rng = np.random.default_rng(5)
    h = np.tanh(rng.standard_normal((B, H))).astype(np.float32)
    mask = inp["mask"].copy()
    mask[0] = 0
    m = wmlib.pack(inp["weights"], Z, H, A, 2, dtype)
    probs, act = wmlib.controller_step(m, _t(inp["z0"]), _t(h), _t(mask), seed=77, step=4, traj0=3)
    torch.cuda.synchronize()
    ref = owm.controller_step(inp["weights"], w.dims, inp["z0"], h, mask, seed=77, step=4,
                              traj0=3, dtype=dtype)
    parity.close(probs.cpu().numpy(), ref["probs"], parity.RTOL[dtype], "probs")
    p = probs.cpu().numpy()
    assert np.all(p[mask == 0] == 0.0)
    a = act.cpu().numpy()
    assert a[0] == -1
    diff = a != ref["action"]
    eps = parity.EPS_TIE[dtype]
    assert np.all(ref["margin"][diff] < eps * (1 + np.abs(ref["top"][diff]))), "non-tie mismatch"
    assert diff.sum() <= 1e-3 * B


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["tiny_rollout", "medium_rollout"])
def test_rollout_fp32_workloads(name):
    w = wl.WORKLOADS[name]
    say("rollout", name)
    inp = wl.make_rollout_inputs(w)
    g = run_rollout(w, inp, trace=True)
    ref = owm.rollout(inp["weights"], w.dims, inp["z0"], inp["mask"], T=w.T, seed=w.seed,
                      tau=w.tau, done_flag=w.done, dtype=w.dtype)
    rec = {}
    diverged = parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=inp["mask"],
                               seed=w.seed, tau=w.tau, dtype=w.dtype, record=rec)
    ties, live = parity.reanchored(w.dims, inp["weights"], inp["mask"], g, seed=w.seed,
                                   tau=w.tau, done_flag=w.done, dtype=w.dtype)
    say(name, "free run", rec, "re-anchored tie mismatches", ties.mismatches, "of", ties.draws,
        "live transitions", live)
    parity.record_ties(name, reanchored_draws=ties.draws, reanchored_mismatches=ties.mismatches,
                       live_transitions=live, **rec)
    assert diverged <= parity.free_run_cap(w.B)
    if w.done:
        assert 0 < g["dones"].sum() < g["dones"].size  # the done head is exercised


@pytest.mark.parametrize("dtype,B,A", [("fp32", 45, 700), ("bf16", 150, 1500)])
def test_rollout_wide_controller(dtype, B, A):
    """Rollouts whose controller has more than 318 logit rows (the wide
    controller kernel), free-running against the oracle and re-anchored."""
    w = wl.Workload("wide", "rollout", B=B, T=4, Z=32, H=256, A=A, K=3, dtype=dtype, seed=31)
    say("rollout wide controller", dtype, B, A)
    inp = wl.make_rollout_inputs(w)
    g = run_rollout(w, inp, trace=True)
    if dtype == "fp32":
        ref = owm.rollout(inp["weights"], w.dims, inp["z0"], inp["mask"], T=w.T, seed=w.seed,
                          tau=w.tau, done_flag=w.done, dtype=w.dtype)
        diverged = parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=inp["mask"],
                                   seed=w.seed, tau=w.tau, dtype=w.dtype)
        assert diverged <= parity.free_run_cap(w.B)
    ties, live = parity.reanchored(w.dims, inp["weights"], inp["mask"], g, seed=w.seed,
                                   tau=w.tau, done_flag=w.done, dtype=w.dtype)
    say("wide: tie mismatches", ties.mismatches, "of", ties.draws, "live", live)
    assert live > 0


def test_nll_workload():
    w = wl.WORKLOADS["nll"]
    say("nll", w)
    d = wl.make_nll_inputs(w)
    m = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    b = wmlib.nll(m, _t(d["z"]), _t(d["actions"]), _t(d["rewards"]), _t(d["dones"]))
    torch.cuda.synchronize()
    ref = owm.nll(d["weights"], w.dims, d["z"], d["actions"], d["rewards"], d["dones"],
                  dtype=w.dtype)
    rt = parity.RTOL[w.dtype]
    parity.close(b.loglik.cpu().numpy(), ref["loglik"], rt, "loglik")
    parity.close(b.reward_se.cpu().numpy(), ref["reward_se"], rt, "reward_se")
    parity.close(b.done_bce.cpu().numpy(), ref["done_bce"], rt, "done_bce")
    parity.close(b.means.cpu().numpy(), ref["means"], rt, "means")
    parity.record_ties("nll", discrete_outputs=0)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,nrows", [("large_rollout", 1024), ("xlarge_rollout", 1024)])
def test_rollout_bf16_workloads_reanchored(name, nrows):
    """Full-size bf16 rollouts in the launch configuration the bench times,
    re-anchored against the oracle on 1024 evenly spread rows (the result of
    a row does not depend on the others)."""
    w = wl.WORKLOADS[name]
    say("rollout", name, "full size with trace")
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    b = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=w.T, seed=w.seed, tau=w.tau,
                      done=w.done, trace=True)
    torch.cuda.synchronize()
    rows = np.unique(np.linspace(0, w.B - 1, nrows).astype(np.int64))
    ri = torch.from_numpy(rows).cuda()
    g = {"z_out": b.z_out[:, ri].cpu().numpy(), "actions": b.actions[:, ri].cpu().numpy(),
         "rewards": b.rewards[:, ri].cpu().numpy(), "dones": b.dones[:, ri].cpu().numpy(),
         "h_trace": b.h_trace[:, ri].cpu().numpy(), "c_trace": b.c_trace[:, ri].cpu().numpy()}
    acts = b.actions.cpu().numpy()
    dones = b.dones.cpu().numpy()
    del b
    torch.cuda.empty_cache()
    say(name, "oracle re-anchored on", rows.size, "rows")
    ties, live = parity.reanchored(w.dims, inp["weights"], inp["mask"][rows], g, seed=w.seed,
                                   tau=w.tau, done_flag=w.done, dtype=w.dtype, traj=rows)
    say(name, "tie mismatches", ties.mismatches, "of", ties.draws, "live", live)
    parity.record_ties(name, reanchored_rows=int(rows.size), reanchored_draws=ties.draws,
                       reanchored_mismatches=ties.mismatches, live_transitions=live)
    # whole-batch invariants: masked actions never taken, frozen pattern sticky
    taken = acts >= 0
    tt, bb = np.nonzero(taken)
    assert np.all(inp["mask"][bb, acts[taken]] == 1)
    first_done = np.where(dones.any(0), dones.argmax(0), w.T)
    for t in range(w.T):
        after = t > first_done
        assert np.all(acts[t, after] == -1) and np.all(dones[t, after] == 1)


def test_rollout_bf16_ragged_wide_tiles():
    """A bf16 batch just past a multiple of the 256-row gate / mixture tiles
    and the 64-row controller tiles (the many-tile configurations), with the
    ragged last tiles among the re-anchored rows."""
    w = wl.WORKLOADS["xlarge_rollout"].replace(B=16384 + 6, T=3)
    say("rollout ragged", w.B, "x", w.T)
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    b = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=w.T, seed=w.seed, tau=w.tau,
                      done=w.done, trace=True)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([np.linspace(0, w.B - 1, 40).astype(np.int64),
                                     np.arange(16384 - 3, w.B), [255, 256, 16383 - 63, 16384 - 64]]))
    ri = torch.from_numpy(rows).cuda()
    g = {k: getattr(b, k)[:, ri].cpu().numpy()
         for k in ("z_out", "actions", "rewards", "dones", "h_trace", "c_trace")}
    del b
    torch.cuda.empty_cache()
    say("ragged: oracle re-anchored on", rows.size, "rows")
    ties, live = parity.reanchored(w.dims, inp["weights"], inp["mask"][rows], g, seed=w.seed,
                                   tau=w.tau, done_flag=w.done, dtype=w.dtype, traj=rows)
    say("ragged: tie mismatches", ties.mismatches, "of", ties.draws, "live", live)
    assert live > 0
