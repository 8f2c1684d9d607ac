"""Variable-length dream rollouts (per-trajectory horizons, zero-padded as
the sequences of section 3.3.1) through the C ABI, on the persistent fp32
path, the multi-launch fp32 path and the bf16 many-tile path:

* against the oracle, re-anchored per step and (fp32) free-running, with
  every step past a horizon checked as padding;
* against the same call without horizons: identical outputs on every
  trajectory's real steps (bit for bit: the same kernels run), and the
  final state and done flags equal to the plain rollout's after each
  trajectory's last real step;
* horizons 0, 1, T, above T and negative.
"""

import os
import sys
from contextlib import contextmanager

import numpy as np
import pytest
import torch

import parity
from oracle import wm as owm
from paper_2205_01435_amd import _lib as wmlib
from paper_2205_01435_amd import workloads as wl

pytestmark = pytest.mark.gpu
KEYS = ("z_out", "actions", "rewards", "dones", "h_T", "c_T", "h_trace", "c_trace")


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


def _np(b, dio=None):
    torch.cuda.synchronize()
    out = {k: getattr(b, k).cpu().numpy() for k in KEYS if getattr(b, k) is not None}
    if dio is not None:
        out["done_io"] = dio.cpu().numpy()
    return out


def _lengths(B, T, seed):
    rng = np.random.default_rng(seed)
    ln = rng.integers(0, T + 1, size=B).astype(np.int32)
    ln[:5] = [0, 1, T, T + 7, -3]
    return ln


CASES = [  # B, T, Z, H, A, K, dtype, persistent
    (100, 9, 32, 256, 20, 4, "fp32", True),
    (100, 9, 32, 256, 20, 4, "fp32", False),
    (70, 6, 24, 80, 33, 3, "bf16", False),
    (4101, 3, 64, 1024, 128, 8, "bf16", False),  # many-tile bf16 configurations, ragged
]


@pytest.mark.parametrize("B,T,Z,H,A,K,dtype,persistent", CASES)
def test_lengths(B, T, Z, H, A, K, dtype, persistent):
    say("lengths", B, T, Z, H, A, K, dtype, "persistent" if persistent else "launches")
    w = wl.Workload("len", "rollout", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype=dtype, seed=B + T)
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], Z, H, A, K, dtype)
    ln = _lengths(B, T, B)
    z0, mask = _t(inp["z0"]), _t(inp["mask"])
    kw = dict(T=T, seed=9, tau=1.2, done=True, trace=True, traj0=3, step0=1)

    def run(**extra):
        dio = torch.zeros(B, dtype=torch.uint8, device="cuda")
        b = wmlib.rollout(m, z0, mask, done_io=dio, **kw, **extra)
        return _np(b, dio)

    if persistent:
        g, full = run(lengths=_t(ln)), run()
    else:
        with launch_path():
            g, full = run(lengths=_t(ln)), run()
    hz = np.clip(ln, 0, T)
    for b in range(B):
        L = hz[b]
        for k in ("actions", "rewards", "dones"):
            np.testing.assert_array_equal(g[k][:L, b], full[k][:L, b], err_msg=f"{k} row {b}")
        np.testing.assert_array_equal(g["z_out"][:L + 1, b], full["z_out"][:L + 1, b])
        np.testing.assert_array_equal(g["h_T"][b], full["h_trace"][L, b])
        np.testing.assert_array_equal(g["c_T"][b], full["c_trace"][L, b])
        assert g["done_io"][b] == (full["dones"][:L, b].any() if L else 0)
    rows = np.unique(np.concatenate([np.arange(min(B, 40)), np.linspace(0, B - 1, 64).astype(np.int64)]))
    sub = {k: g[k][:, rows] for k in ("z_out", "actions", "rewards", "dones", "h_trace", "c_trace")}
    ties, live = parity.reanchored(w.dims, inp["weights"], inp["mask"][rows], sub, seed=9, tau=1.2,
                                   done_flag=True, dtype=dtype, traj=3 + rows, step0=1, lengths=ln[rows])
    say("ties", ties.mismatches, "of", ties.draws, "live", live)
    if dtype == "fp32":
        ref = owm.rollout(inp["weights"], w.dims, inp["z0"], inp["mask"], T=T, seed=9, tau=1.2,
                          done_flag=True, traj0=3, step0=1, lengths=ln)
        div = parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=inp["mask"], seed=9,
                              tau=1.2, traj=3 + np.arange(B), step0=1, lengths=ln)
        assert div <= parity.free_run_cap(B)
        np.testing.assert_array_equal(g["done_io"], ref["done_T"])
