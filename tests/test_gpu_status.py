"""Device-side status of the C ABI calls (on an MI355X):

* WM_FLAG_CHECK: valid device data passes and gives the same outputs bit for
  bit as a call without the flag; a mask byte other than 0/1 (rollout), an
  action outside [0, A) u {-1, -2} or a done byte other than 0/1 inside a
  sequence (NLL pass, training gradient) returns WM_ERR_INVALID_ARG before any
  output is computed; the same values at padded steps are not checked.
* The persistent kernels' error word: with WM_FLAG_TEST_ABORT the host sets
  it before the launch (no kernel is made to fail or wait); every work-group
  leaves at its first wait and the kernel ends normally; wm_workspace_status
  reports WM_ERR_HIP, and so does the call itself under WM_FLAG_CHECK.  The
  next call on the same workspace starts clean and matches a fresh run.
"""

import sys

import numpy as np
import pytest
import torch

from paper_2205_01435_amd import _lib as wmlib
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


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _launches(prefix, fn):
    wmlib.profile_reset()
    wmlib.profile_enable(prefix)
    try:
        out = fn()
        torch.cuda.synchronize()
        return out, wmlib.profile_read(prefix)[1]
    finally:
        wmlib.profile_enable(None)
        wmlib.profile_reset()


ROLL_KEYS = ("z_out", "actions", "rewards", "dones", "h_T", "c_T")


def _np(b):
    torch.cuda.synchronize()
    return {k: getattr(b, k).cpu().numpy() for k in ROLL_KEYS}


@pytest.mark.parametrize("dtype,B,H", [("fp32", 40, 256), ("bf16", 70, 128)])
def test_check_flag_rollout(dtype, B, H):
    """fp32 at H 256 runs the persistent kernel, bf16 the multi-launch path."""
    say("check rollout", dtype, B, H)
    w = wl.Workload("s", "rollout", B=B, T=5, Z=16, H=H, A=12, K=3, dtype=dtype, seed=41)
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, dtype)
    z0, mask = _t(inp["z0"]), _t(inp["mask"])
    plain = _np(wmlib.rollout(m, z0, mask, T=w.T, seed=3, done=True))
    checked = _np(wmlib.rollout(m, z0, mask, T=w.T, seed=3, done=True, check=True))
    for k in ROLL_KEYS:
        np.testing.assert_array_equal(checked[k], plain[k], err_msg=k)
    bad = inp["mask"].copy()
    bad[B - 1, 3] = 2
    with pytest.raises(wmlib.WmError) as ei:
        wmlib.rollout(m, z0, _t(bad), T=w.T, seed=3, done=True, check=True)
    assert ei.value.status == wmlib.WM_ERR_INVALID_ARG and "1 precondition" in str(ei.value)
    # per-step masks: a bad byte in the last step's slice
    sm = np.broadcast_to(inp["mask"], (w.T, B, w.A)).copy()
    sm[w.T - 1, 0, 0] = 255
    with pytest.raises(wmlib.WmError) as ei:
        wmlib.rollout(m, z0, _t(sm), T=w.T, seed=3, done=True, check=True)
    assert ei.value.status == wmlib.WM_ERR_INVALID_ARG


def test_check_flag_nll_and_grad():
    w = wl.Workload("s", "nll", B=33, T=6, Z=16, H=64, A=9, K=2, dtype="fp32", seed=42)
    d = wl.make_nll_inputs(w)
    m = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, "fp32")
    lengths = np.full(w.B, w.T, np.int32)
    lengths[5] = 2
    a = d["actions"].copy()
    a[0, 1], a[1, 2] = -1, -2  # the codes a rollout emits: allowed
    a[4, 5] = 1000  # padded step of sequence 5: not checked
    args = [_t(d["z"]), _t(a), _t(d["rewards"]), _t(d["dones"]), _t(lengths)]
    plain = wmlib.nll(m, *args)
    torch.cuda.synchronize()
    p = {k: getattr(plain, k).clone() for k in ("loglik", "reward_se", "done_bce", "means")}
    checked = wmlib.nll(m, *args, check=True)
    for k in p:
        assert torch.equal(p[k], getattr(checked, k)), k
    wmlib.nll_grad(m, *args, check=True)
    for t, b, v in ((2, 7, w.A), (3, 8, -3)):
        bad = a.copy()
        bad[t, b] = v
        with pytest.raises(wmlib.WmError) as ei:
            wmlib.nll(m, args[0], _t(bad), *args[2:], check=True)
        assert ei.value.status == wmlib.WM_ERR_INVALID_ARG
        with pytest.raises(wmlib.WmError) as ei:
            wmlib.nll_grad(m, args[0], _t(bad), *args[2:], check=True)
        assert ei.value.status == wmlib.WM_ERR_INVALID_ARG
    dn = d["dones"].copy()
    dn[0, 0] = 2
    with pytest.raises(wmlib.WmError) as ei:
        wmlib.nll(m, *args[:3], _t(dn), args[4], check=True)
    assert "1 precondition" in str(ei.value)


def test_abort_word_rollout_persistent():
    w = wl.WORKLOADS["medium_rollout"]
    say("abort word: persistent rollout", w.B, w.T)
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = _t(inp["z0"]), _t(inp["mask"])
    bufs = wmlib.RolloutBuffers(m, w.B, w.T)
    run = lambda **kw: wmlib.rollout(m, z0, mask, T=w.T, seed=w.seed, done=True, bufs=bufs, **kw)  # noqa: E731
    _, n = _launches("persist", lambda: run(extra_flags=wmlib.WM_FLAG_TEST_ABORT))
    assert n == 1, "the persistent kernel did not run"
    with pytest.raises(wmlib.WmError) as ei:
        wmlib.status(bufs)
    assert ei.value.status == wmlib.WM_ERR_HIP and "timed out" in str(ei.value)
    with pytest.raises(wmlib.WmError) as ei:
        run(extra_flags=wmlib.WM_FLAG_TEST_ABORT, check=True)
    assert ei.value.status == wmlib.WM_ERR_HIP
    # the next call on the same workspace starts clean
    run()
    wmlib.status(bufs)
    got = _np(bufs)
    fresh = _np(wmlib.rollout(m, z0, mask, T=w.T, seed=w.seed, done=True))
    for k in ROLL_KEYS:
        np.testing.assert_array_equal(got[k], fresh[k], err_msg=k)


def test_abort_word_nll_persistent():
    w = wl.Workload("s", "nll", B=100, T=5, Z=32, H=256, A=9, K=2, dtype="fp32", seed=43)
    say("abort word: persistent NLL recurrence", w.B, w.T)
    d = wl.make_nll_inputs(w)
    m = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, "fp32")
    args = [_t(d[k]) for k in ("z", "actions", "rewards", "dones")]
    bufs = wmlib.NllBuffers(m, w.B, w.T)
    _, n = _launches("nll_persist", lambda: wmlib.nll(m, *args, bufs=bufs, extra_flags=wmlib.WM_FLAG_TEST_ABORT))
    assert n == 1, "the persistent recurrence did not run"
    with pytest.raises(wmlib.WmError) as ei:
        wmlib.status(bufs)
    assert ei.value.status == wmlib.WM_ERR_HIP
    ref = wmlib.nll(m, *args)
    wmlib.nll(m, *args, bufs=bufs)
    wmlib.status(bufs)
    assert torch.equal(bufs.loglik, ref.loglik) and torch.equal(bufs.means, ref.means)
