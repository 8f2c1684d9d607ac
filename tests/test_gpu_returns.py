"""GPU parity of the return scan (wm_returns, through the C ABI) against the
oracle, element by element, on seeded inputs: short and long horizons (one
and several windows of the kernel), ragged batches, gamma 0 and 1, lambda 0,
0.95 and 1, full xlarge-rollout shapes, and a real rollout's outputs."""

import sys

import numpy as np
import pytest
import torch

import parity
from oracle import returns as oret
from paper_2205_01435_amd import _lib as wmlib
from paper_2205_01435_amd import workloads as wl

pytestmark = pytest.mark.gpu
RTOL = parity.RTOL["fp32"]


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    wmlib.load()
    yield


def _inputs(T, B, seed, pdone=0.05, with_values=False):
    rng = np.random.default_rng(seed)
    r = rng.normal(size=(T, B)).astype(np.float32)
    d = (rng.random((T, B)) < pdone).astype(np.uint8)
    V = rng.normal(size=(T + 1, B)).astype(np.float32) if with_values else None
    return r, d, V


def _run(r, d, V, gamma, lam):
    t = lambda x: None if x is None else torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    ret, adv = wmlib.returns(t(r), t(d), gamma, values=t(V), lam=lam)
    torch.cuda.synchronize()
    return ret.cpu().numpy(), None if adv is None else adv.cpu().numpy()


CASES = [  # T, B, gamma, lam, values
    (1, 1, 0.99, 1.0, False), (16, 1, 0.99, 1.0, False), (17, 5, 0.9, 1.0, True),
    (20, 16, 0.99, 0.95, True), (50, 256, 0.99, 1.0, False), (64, 16384, 0.99, 0.95, True),
    (100, 4096, 0.97, 1.0, False), (300, 33, 0.995, 0.9, True), (257, 70, 1.0, 1.0, False),
    (40, 100, 0.0, 0.5, True), (33, 65, 0.8, 0.0, True), (1000, 3, 0.999, 0.95, True),
]


@pytest.mark.parametrize("T,B,gamma,lam,with_values", CASES)
def test_returns_parity(T, B, gamma, lam, with_values):
    say("returns", T, B, gamma, lam, with_values)
    r, d, V = _inputs(T, B, seed=T * 7919 + B, with_values=with_values)
    ret, adv = _run(r, d, V, gamma, lam)
    ref, ref_adv = oret.returns(r, d, gamma, values=V, lam=lam)
    parity.close(ret, ref, RTOL, "returns")
    if with_values:
        parity.close(adv, ref_adv, RTOL, "advantages")
    else:
        assert adv is None


def test_returns_of_a_rollout():
    """The scan reads a rollout's outputs as they are (frozen steps included)."""
    w = wl.WORKLOADS["medium_rollout"]
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    b = wmlib.rollout(m, torch.from_numpy(inp["z0"]).cuda(), torch.from_numpy(inp["mask"]).cuda(),
                      T=w.T, seed=w.seed, tau=w.tau, done=w.done)
    ret, _ = wmlib.returns(b.rewards, b.dones, 0.99)
    torch.cuda.synchronize()
    r, d = b.rewards.cpu().numpy(), b.dones.cpu().numpy()
    assert d.any(), "the workload's done head fires"
    ref, _ = oret.returns(r, d, 0.99)
    parity.close(ret.cpu().numpy(), ref, RTOL, "returns")


def test_returns_argument_errors():
    r = torch.zeros((4, 3), dtype=torch.float32, device="cuda")
    d = torch.zeros((4, 3), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(r)
    lib = wmlib.load()
    p = lambda x: None if x is None else __import__("ctypes").c_void_p(x.data_ptr())  # noqa: E731
    s = wmlib._stream()
    assert lib.wm_returns(3, 4, p(r), p(d), None, 1.5, 1.0, p(out), None, s) == -1  # gamma > 1
    assert lib.wm_returns(3, 4, p(r), p(d), None, 0.9, -0.1, p(out), None, s) == -1  # lambda < 0
    assert lib.wm_returns(3, 4, p(r), p(d), None, 0.9, 1.0, p(out), p(out), s) == -1  # adv without V
    assert lib.wm_returns(3, 4, None, p(d), None, 0.9, 1.0, p(out), None, s) == -1
    assert lib.wm_returns(-1, 4, p(r), p(d), None, 0.9, 1.0, p(out), None, s) == -1
    assert lib.wm_returns(0, 4, None, None, None, 0.9, 1.0, None, None, s) == 0   # empty: no-op
    assert lib.wm_returns(3, 0, None, None, None, 0.9, 1.0, None, None, s) == 0
