"""wm_rollout_noalloc (the rollout on the library's static device scratch)
against wm_rollout with a caller workspace, through the C ABI: identical
outputs bit for bit (the same kernels run), on two calls in a row, the
second with a smaller input, on the persistent path (fp32) and the
multi-launch path (bf16); a batch whose workspace exceeds the static scratch
is refused with WM_ERR_UNSUPPORTED."""

import sys

import numpy as np
import pytest
import torch

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


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _pair(w, seed, trace):
    inp = wl.make_rollout_inputs(w)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = _t(inp["z0"]), _t(inp["mask"])
    kw = dict(T=w.T, seed=seed, tau=1.3, done=True, trace=trace, traj0=5, step0=2)
    ref = wmlib.rollout(m, z0, mask, **kw)
    got = wmlib.rollout(m, z0, mask, noalloc=True, **kw)
    torch.cuda.synchronize()
    for k in KEYS:
        a, b = getattr(got, k), getattr(ref, k)
        if b is None:
            continue
        assert torch.equal(a, b), f"{w.name} {k}"
    assert bool((ref.actions >= 0).any())


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_noalloc_matches_workspace_call(dtype):
    big = wl.WORKLOADS["medium_rollout"].replace(name="first", dtype=dtype)
    small = wl.WORKLOADS["tiny_rollout"].replace(name="second", dtype=dtype, T=9)
    say("noalloc", dtype, "B", big.B, "then B", small.B)
    _pair(big, 11, trace=False)
    _pair(small, 12, trace=True)


def test_noalloc_refuses_beyond_the_scratch():
    w = wl.WORKLOADS["xlarge_rollout"]
    dims = wmlib.make_dims(w.Z, w.H, w.A, w.K, w.dtype)
    need = wmlib.workspace_bytes(dims, w.B, w.T, wmlib.WS_ROLLOUT)
    assert need > 64 << 20
    inp = wl.make_rollout_inputs(w.replace(B=8))
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0 = torch.zeros((w.B, w.Z), dtype=torch.float32, device="cuda")
    mask = torch.ones((w.B, w.A), dtype=torch.uint8, device="cuda")
    with pytest.raises(wmlib.WmError) as ei:
        wmlib.rollout(m, z0, mask, T=2, seed=1, noalloc=True)
    assert ei.value.status == wmlib.WM_ERR_UNSUPPORTED and "static scratch" in str(ei.value)
