"""GPU parity of the optimiser step (wm_adam_step, through the C ABI)
against the oracle's Adam, element by element, over three steps with
changing gradients; a size that is not a multiple of four exercises the
tail; argument errors."""

import numpy as np
import pytest
import torch

import parity
from oracle import train as otr
from paper_2205_01435_amd import _lib as wmlib

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    wmlib.load()
    yield


@pytest.mark.parametrize("n,lr", [(3, 1e-2), (1000003, 3e-4), (4096, 0.0)])
def test_adam_parity(n, lr):
    rng = np.random.default_rng(n)
    p = rng.normal(size=n).astype(np.float32)
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    P = dev(p)
    M = torch.zeros(n, dtype=torch.float32, device="cuda")
    V = torch.zeros_like(M)
    ref = {"x": p.astype(np.float64)}
    st = {}
    for step in (1, 2, 3):
        g = (rng.normal(size=n) * 10.0 ** rng.uniform(-3, 1, size=n)).astype(np.float32)
        wmlib.adam_step(P, dev(g), M, V, step, lr)
        ref = otr.adam_step(ref, {"x": g}, st, lr)
        torch.cuda.synchronize()
        parity.close(P.cpu().numpy(), ref["x"], parity.RTOL["fp32"], f"params step {step}")
        parity.close(M.cpu().numpy(), st["m_x"], parity.RTOL["fp32"], f"m step {step}")
        parity.close(V.cpu().numpy(), st["v_x"], parity.RTOL["fp32"], f"v step {step}")


def test_adam_argument_errors():
    x = torch.zeros(8, dtype=torch.float32, device="cuda")
    with pytest.raises(wmlib.WmError):
        wmlib.adam_step(x, x, x, x, 0, 1e-3)          # steps count from 1
    with pytest.raises(wmlib.WmError):
        wmlib.adam_step(x, x, x, x, 1, 1e-3, beta1=1.0)
    with pytest.raises(wmlib.WmError):
        wmlib.adam_step(x, x, x, x, 1, float("nan"))
