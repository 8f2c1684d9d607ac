"""The vectorised oracle against the brute-force scalar loops (tiny shapes)."""

import numpy as np
import pytest

from oracle import brute, wm
from paper_2205_01435_amd import workloads as wl

SHAPES = [
    dict(B=3, T=4, Z=2, H=3, A=4, K=2),
    dict(B=3, T=4, Z=2, H=3, A=4, K=1),
    dict(B=4, T=3, Z=4, H=5, A=3, K=3),
]


def _case(shape, dtype, seed, done_bias=None):
    w = wl.Workload("t", "rollout", dtype=dtype, seed=seed, mask_p=0.5, **shape)
    d = wl.make_rollout_inputs(w)
    wts = d["weights"]
    rng = np.random.default_rng(seed + 100)
    wts["b_g"] = (rng.normal(size=wts["b_g"].shape) * 0.5).astype(np.float32)
    wts["b_m"] = (rng.normal(size=wts["b_m"].shape) * 0.5).astype(np.float32)
    wts["b_c"] = (rng.normal(size=wts["b_c"].shape) * 0.5).astype(np.float32)
    if done_bias is not None:
        wts["b_d"] = np.float32(done_bias)
    return w, d


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_rollout_matches_brute(shape, dtype):
    w, d = _case(shape, dtype, seed=11, done_bias=-1.0)
    mask = d["mask"].copy()
    mask[-1] = 0  # a row with no valid action
    done0 = np.zeros(w.B, np.uint8)
    done0[0] = 1  # a row already finished
    rng = np.random.default_rng(1)
    h0 = rng.normal(size=(w.B, w.H)).astype(np.float32) * 0.5
    c0 = rng.normal(size=(w.B, w.H)).astype(np.float32) * 0.5
    kw = dict(T=w.T, seed=99, tau=1.3, done_flag=True, dtype=dtype, traj0=5, step0=2)
    v = wm.rollout(d["weights"], w.dims, d["z0"], mask, h0=h0, c0=c0, done0=done0, **kw)
    b = brute.rollout(d["weights"], w.dims, d["z0"], mask, h0=h0, c0=c0, done0=done0, **kw)
    np.testing.assert_array_equal(v["actions"], np.array(b["actions"]))
    np.testing.assert_array_equal(v["dones"], np.array(b["dones"]))
    np.testing.assert_array_equal(v["done_T"], np.array(b["done_T"]))
    np.testing.assert_allclose(v["z_out"], np.array(b["z_out"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v["rewards"], np.array(b["rewards"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v["h_T"], np.array(b["h_T"]), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(v["c_T"], np.array(b["c_T"]), rtol=1e-12, atol=1e-12)
    # the case exercises every branch: frozen input row, empty mask, live rows
    assert np.all(v["actions"][:, 0] == -1) and np.all(v["actions"][:, -1] == -1)
    assert np.any(v["actions"] >= 0)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_controller_step_matches_brute(dtype):
    w, d = _case(SHAPES[2], dtype, seed=12)
    rng = np.random.default_rng(2)
    h = rng.normal(size=(w.B, w.H)).astype(np.float32)
    mask = d["mask"].copy()
    mask[1] = 0
    v = wm.controller_step(d["weights"], w.dims, d["z0"], h, mask, seed=7, step=3, traj0=2,
                           dtype=dtype)
    b = brute.controller_step(d["weights"], w.dims, d["z0"], h, mask, seed=7, step=3, traj0=2,
                              dtype=dtype)
    np.testing.assert_array_equal(v["action"], np.array(b["action"]))
    np.testing.assert_allclose(v["probs"], np.array(b["probs"]), rtol=1e-12, atol=1e-15)
    assert v["action"][1] == -1


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", SHAPES)
def test_nll_matches_brute(shape, dtype):
    w = wl.Workload("t", "nll", dtype=dtype, seed=13, **shape)
    d = wl.make_nll_inputs(w)
    lengths = np.array([w.T, 1, 0, 2][:w.B])
    acts = d["actions"].copy()
    acts[0, 0] = -1  # a step with no action: zero one-hot column
    for lens in (None, lengths):
        v = wm.nll(d["weights"], w.dims, d["z"], acts, d["rewards"], d["dones"], lengths=lens,
                   dtype=dtype)
        b = brute.nll(d["weights"], w.dims, d["z"], acts, d["rewards"], d["dones"],
                      lengths=lens, dtype=dtype)
        for k in ("loglik", "reward_se", "done_bce"):
            np.testing.assert_allclose(v[k], np.array(b[k]), rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(v["means"], np.array(b["means"]), rtol=1e-11, atol=1e-12)
