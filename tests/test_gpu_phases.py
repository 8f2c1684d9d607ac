"""Phase stamps of the persistent kernels (wm_profile_phases): the stamped
launch computes the same outputs bit for bit, and the per-step slots are
positive and add up to about the step (the barrier slots and the work
slots tile each step, apart from the skew between work-groups)."""

import sys

import numpy as np
import pytest
import torch

from paper_2205_01435_amd import _lib as wmlib
from paper_2205_01435_amd import phases
from paper_2205_01435_amd import workloads as wl

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    wmlib.load()
    yield
    wmlib.profile_phases(False)


def test_stamped_rollout_is_unchanged():
    w = wl.WORKLOADS["tiny_rollout"]
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = torch.from_numpy(inp["z0"]).cuda(), torch.from_numpy(inp["mask"]).cuda()

    def run():
        b = wmlib.rollout(m, z0, mask, T=w.T, seed=3, done=True, trace=True)
        torch.cuda.synchronize()
        return {k: getattr(b, k).cpu().numpy() for k in ("z_out", "actions", "rewards", "dones", "h_trace")}

    plain = run()
    wmlib.profile_phases(True)
    try:
        stamped = run()
        r = wmlib.profile_phases_read()
    finally:
        wmlib.profile_phases(False)
    for k in plain:
        np.testing.assert_array_equal(plain[k], stamped[k], err_msg=k)
    say("phases", {k: round(v, 3) for k, v in r.items()})
    assert r["T"] == w.T
    for k in wmlib.PHASE_SLOTS[1:]:
        if k.startswith("ctrl"):
            assert r[k] == 0, k  # the controller runs inside the gate phase
        else:
            assert r[k] > 0, k
    tiles = sum(r[k] for k in ("gates", "gates_barrier", "mdn", "mdn_barrier"))
    assert 0.5 * r["step"] < tiles < 1.5 * r["step"]
    assert wmlib.profile_phases_read()["T"] == w.T  # the last stamped launch, read again
    wmlib.profile_phases(True)
    assert wmlib.profile_phases_read()["T"] == 0  # switching on forgets it
    wmlib.profile_phases(False)


@pytest.mark.parametrize("name", ["medium_rollout", "nll"])
def test_phase_summary(name):
    res = phases.measure(name, calls=3, warmup=1)
    say(name, {k: round(v, 3) for k, v in res.items()})
    assert res["T"] == wl.WORKLOADS[name].T and res["step"] > 0 and res["gates"] > 0
    assert "| gates |" in phases.summary(name, res, 3)
