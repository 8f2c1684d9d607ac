"""GPU parity of the rollout's optional variants against the oracle, through
the C ABI: the sigma temperature (WM_FLAG_SIGMA_TAU) on the persistent path,
the multi-launch path (fp32 and bf16, including the many-tile bf16
configurations), re-anchored per step."""

import os
import sys
from contextlib import contextmanager

import numpy as np
import pytest
import torch

import parity
from paper_2205_01435_amd import _lib as wmlib
from paper_2205_01435_amd import workloads as wl

pytestmark = pytest.mark.gpu
KEYS = ("z_out", "actions", "rewards", "dones", "h_trace", "c_trace")


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    wmlib.load()
    yield


@contextmanager
def launch_path():
    old = os.environ.get("WM_PERSISTENT")
    os.environ["WM_PERSISTENT"] = "0"
    try:
        yield
    finally:
        if old is None:
            del os.environ["WM_PERSISTENT"]
        else:
            os.environ["WM_PERSISTENT"] = old


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


# (B, T, Z, H, A, K, dtype, path, rows compared)
SIGMA = [
    (37, 4, 24, 256, 20, 3, "fp32", "persistent", None),
    (37, 4, 24, 256, 20, 3, "fp32", "launch", None),
    (300, 3, 64, 512, 64, 8, "fp32", "launch", None),
    (64, 3, 16, 128, 8, 5, "bf16", "launch", None),
    (4096 + 5, 2, 128, 1024, 256, 8, "bf16", "launch", 48),  # 256-row gate and mixture tiles
]


@pytest.mark.parametrize("B,T,Z,H,A,K,dtype,path,nrows", SIGMA)
def test_sigma_temperature(B, T, Z, H, A, K, dtype, path, nrows):
    say("sigma temperature", B, T, Z, H, A, K, dtype, path)
    w = wl.Workload("v", "rollout", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype=dtype, seed=B + K,
                    mask_p=0.4)
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], Z, H, A, K, dtype)
    args = dict(T=T, seed=23, tau=1.7, done=True, trace=True, sigma_tau=True)
    if path == "launch":
        with launch_path():
            b = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), **args)
    else:
        wmlib.profile_reset()
        wmlib.profile_enable("persist")
        try:
            b = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), **args)
            torch.cuda.synchronize()
            _, n = wmlib.profile_read("persist")
        finally:
            wmlib.profile_enable(None)
            wmlib.profile_reset()
        assert n == 1, "the persistent kernel did not run"
    torch.cuda.synchronize()
    rows = np.arange(B) if nrows is None else np.unique(
        np.concatenate([np.linspace(0, B - 1, nrows).astype(np.int64), np.arange(B - 5, B)]))
    ri = torch.from_numpy(rows).cuda()
    g = {k: getattr(b, k)[:, ri].cpu().numpy() for k in KEYS}
    ties, live = parity.reanchored(w.dims, inp["weights"], inp["mask"][rows], g, seed=23, tau=1.7,
                                   done_flag=True, dtype=dtype, traj=rows, sigma_tau=True)
    say("ties", ties.mismatches, "of", ties.draws, "live", live)
    assert live > 0
    # the flag changes the draws: without it the same seed gives other latents
    plain = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=1, seed=23, tau=1.7, done=True)
    torch.cuda.synchronize()
    assert not np.allclose(plain.z_out[1].cpu().numpy()[rows], g["z_out"][1])


# (B, T, Z, H, A, K, dtype, path, rows compared)
STEPMASK = [
    (37, 5, 24, 256, 20, 3, "fp32", "persistent", None),
    (37, 5, 24, 256, 20, 3, "fp32", "launch", None),
    (64, 4, 16, 128, 40, 5, "bf16", "launch", None),
    (16384 + 6, 2, 128, 1024, 256, 8, "bf16", "launch", 40),  # 64-row controller tiles
]


@pytest.mark.parametrize("B,T,Z,H,A,K,dtype,path,nrows", STEPMASK)
def test_per_step_masks(B, T, Z, H, A, K, dtype, path, nrows):
    say("per-step masks", B, T, Z, H, A, K, dtype, path)
    w = wl.Workload("v", "rollout", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype=dtype, seed=B + A,
                    mask_p=0.4)
    inp = wl.make_rollout_inputs(w)
    rng = np.random.default_rng(B)
    sm = (rng.random((T, B, A)) < 0.3).astype(np.uint8)
    sm[np.arange(T)[:, None], np.arange(B)[None, :], rng.integers(0, A, size=(T, B))] = 1
    sm[1, B // 3] = 0  # a row that runs out of valid actions at step 1
    m = wmlib.pack(inp["weights"], Z, H, A, K, dtype)
    args = dict(T=T, seed=29, tau=1.0, done=True, trace=True)
    if path == "launch":
        with launch_path():
            b = wmlib.rollout(m, _t(inp["z0"]), _t(sm), **args)
    else:
        wmlib.profile_reset()
        wmlib.profile_enable("persist")
        try:
            b = wmlib.rollout(m, _t(inp["z0"]), _t(sm), **args)
            torch.cuda.synchronize()
            _, n = wmlib.profile_read("persist")
        finally:
            wmlib.profile_enable(None)
            wmlib.profile_reset()
        assert n == 1, "the persistent kernel did not run"
    torch.cuda.synchronize()
    acts = b.actions.cpu().numpy()
    tt, bb = np.nonzero(acts >= 0)
    assert np.all(sm[tt, bb, acts[tt, bb]] == 1), "an action invalid under its step's mask"
    assert acts[1, B // 3] == -1 and np.all(acts[2:, B // 3] == -1)
    rows = np.arange(B) if nrows is None else np.unique(
        np.concatenate([np.linspace(0, B - 1, nrows).astype(np.int64), np.arange(B - 6, B), [B // 3]]))
    ri = torch.from_numpy(rows).cuda()
    g = {k: getattr(b, k)[:, ri].cpu().numpy() for k in KEYS}
    ties, live = parity.reanchored(w.dims, inp["weights"], sm[:, rows], g, seed=29, tau=1.0,
                                   done_flag=True, dtype=dtype, traj=rows)
    say("ties", ties.mismatches, "of", ties.draws, "live", live)
    assert live > 0


def test_mask_shape_is_checked():
    w = wl.Workload("v", "rollout", B=4, T=3, Z=8, H=16, A=5, K=2, dtype="fp32", seed=1)
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, "fp32")
    with pytest.raises(ValueError):
        wmlib.rollout(m, _t(inp["z0"]), _t(np.ones((2, 4, 5), np.uint8)), T=3, seed=1)
