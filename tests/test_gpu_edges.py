"""GPU edge cases: ragged and degenerate shapes, resume, batch-subset
invariance, determinism, padding, limits and error paths (through the C ABI)."""

import sys

import numpy as np
import pytest
import torch

import parity
from oracle import wm as owm
from paper_2205_01435_amd import _lib as wmlib
from paper_2205_01435_amd import workloads as wl

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-edge]", *a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    wmlib.load()
    yield


def _t(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def _np(b):
    keys = ("z_out", "actions", "rewards", "dones", "h_T", "c_T", "h_trace", "c_trace")
    return {k: getattr(b, k).cpu().numpy() for k in keys if getattr(b, k) is not None}


def _case(B, T, Z, H, A, K, dtype, seed=9, mask_p=0.4, bias=True):
    w = wl.Workload("e", "rollout", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype=dtype, seed=seed,
                    mask_p=mask_p)
    inp = wl.make_rollout_inputs(w)
    if bias:
        rng = np.random.default_rng(seed)
        for k in ("b_g", "b_m", "b_c"):
            inp["weights"][k] = (0.3 * rng.standard_normal(inp["weights"][k].shape)).astype(np.float32)
    return w, inp


RAGGED = [
    (37, 5, 8, 48, 37, 3, "fp32"),
    (37, 5, 8, 48, 37, 3, "bf16"),
    (5, 3, 16, 16, 1, 1, "fp32"),
    (70, 4, 24, 80, 130, 8, "fp32"),
    (70, 4, 24, 80, 130, 8, "bf16"),
    (33, 3, 16, 64, 1000, 2, "fp32"),
    (17, 2, 8, 32, 2048, 4, "bf16"),
    (129, 3, 40, 112, 7, 6, "fp32"),
    (20, 2, 1024, 64, 8, 2, "fp32"),   # the widest latent the library takes
    (20, 2, 1024, 64, 8, 2, "bf16"),
    (9, 2, 8, 2048, 3, 1, "fp32"),     # a wide hidden state: 8192 gate rows
    (9, 2, 8, 2048, 3, 1, "bf16"),
]


@pytest.mark.parametrize("B,T,Z,H,A,K,dtype", RAGGED)
def test_ragged_shapes_reanchored(B, T, Z, H, A, K, dtype):
    say("ragged", B, T, Z, H, A, K, dtype)
    w, inp = _case(B, T, Z, H, A, K, dtype)
    mask = inp["mask"].copy()
    mask[B // 2] = 0  # a row without a valid action
    m = wmlib.pack(inp["weights"], Z, H, A, K, dtype)
    b = wmlib.rollout(m, _t(inp["z0"]), _t(mask), T=T, seed=31, tau=1.3, done=True, trace=True)
    torch.cuda.synchronize()
    g = _np(b)
    ties, live = parity.reanchored(w.dims, inp["weights"], mask, g, seed=31, tau=1.3,
                                   done_flag=True, dtype=dtype)
    assert g["actions"][0, B // 2] == -1 and np.all(g["dones"][:, B // 2] == 1)
    if dtype == "fp32":
        ref = owm.rollout(inp["weights"], w.dims, inp["z0"], mask, T=T, seed=31, tau=1.3,
                          done_flag=True, dtype=dtype)
        assert parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=mask, seed=31,
                               tau=1.3, dtype=dtype) <= parity.free_run_cap(B)


# Staged controller tiles with one or two 64-output blocks (more than 1024
# rows, at most 126 actions), on four and eight waves; the last row tile is
# ragged.  nrows: rows re-anchored against the oracle (None: all).
FEW_ACTIONS = [
    (2048 + 7, 3, 32, 256, 60, 3, "bf16", None),   # 32-row tiles, one output block
    (2048 + 7, 3, 32, 256, 100, 3, "bf16", None),  # 32-row tiles, two output blocks
    (2048 + 7, 3, 32, 256, 100, 3, "fp32", None),  # the same on the fp32 core
    (16384 + 3, 2, 32, 128, 60, 2, "bf16", 48),    # 64-row tiles
]


@pytest.mark.parametrize("B,T,Z,H,A,K,dtype,nrows", FEW_ACTIONS)
def test_few_action_controller_tiles(B, T, Z, H, A, K, dtype, nrows, monkeypatch):
    say("few-action controller tiles", B, T, Z, H, A, K, dtype)
    monkeypatch.setenv("WM_PERSISTENT", "0")  # the multi-launch kernels
    w, inp = _case(B, T, Z, H, A, K, dtype)
    mask = inp["mask"].copy()
    mask[B - 2] = 0  # a row without a valid action, in the ragged tile
    m = wmlib.pack(inp["weights"], Z, H, A, K, dtype)
    b = wmlib.rollout(m, _t(inp["z0"]), _t(mask), T=T, seed=37, tau=1.0, done=True, trace=True)
    torch.cuda.synchronize()
    rows = np.arange(B) if nrows is None else np.unique(
        np.concatenate([np.linspace(0, B - 1, nrows).astype(np.int64), np.arange(B - 6, B)]))
    ri = torch.from_numpy(rows).cuda()
    keys = ("z_out", "actions", "rewards", "dones", "h_trace", "c_trace")
    g = {k: getattr(b, k)[:, ri].cpu().numpy() for k in keys}
    del b
    ties, live = parity.reanchored(w.dims, inp["weights"], mask[rows], g, seed=37, tau=1.0,
                                   done_flag=True, dtype=dtype, traj=rows)
    say("ties", ties.mismatches, "of", ties.draws, "live", live)
    assert live > 0
    k = int(np.searchsorted(rows, B - 2))
    assert g["actions"][0, k] == -1 and np.all(g["dones"][:, k] == 1)


def test_resume_and_state_inputs_bit_exact():
    """rollout(T1) then rollout(T2, step0=T1, state) equals rollout(T1+T2)."""
    w, inp = _case(48, 7, 16, 64, 9, 3, "fp32")
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = _t(inp["z0"]), _t(inp["mask"])
    full = _np(wmlib.rollout(m, z0, mask, T=7, seed=4, done=True))
    dio = torch.zeros(48, dtype=torch.uint8, device="cuda")
    a = wmlib.rollout(m, z0, mask, T=3, seed=4, done=True, done_io=dio)
    torch.cuda.synchronize()
    na = _np(a)
    b = wmlib.rollout(m, a.z_out[3].contiguous(), mask, T=4, seed=4, done=True, step0=3,
                      h0=a.h_T, c0=a.c_T, done_io=dio)
    torch.cuda.synchronize()
    nb = _np(b)
    for k in ("actions", "rewards", "dones"):
        np.testing.assert_array_equal(np.concatenate([na[k], nb[k]]), full[k], err_msg=k)
    np.testing.assert_array_equal(np.concatenate([na["z_out"], nb["z_out"][1:]]), full["z_out"])
    np.testing.assert_array_equal(nb["h_T"], full["h_T"])
    np.testing.assert_array_equal(nb["c_T"], full["c_T"])
    # done_io out = done after the last step
    np.testing.assert_array_equal(dio.cpu().numpy(), (full["dones"][-1] != 0).astype(np.uint8))


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_batch_subset_and_determinism(dtype):
    w, inp = _case(200, 6, 32, 128, 20, 4, dtype)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    full = _np(wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=6, seed=8, done=True))
    again = _np(wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=6, seed=8, done=True))
    for k in full:
        np.testing.assert_array_equal(full[k], again[k], err_msg=f"run-to-run {k}")
    lo, hi = 37, 151
    sub = _np(wmlib.rollout(m, _t(inp["z0"][lo:hi]), _t(inp["mask"][lo:hi]), T=6, seed=8,
                            done=True, traj0=lo))
    for k in ("actions", "dones", "rewards", "z_out"):
        np.testing.assert_array_equal(sub[k], full[k][:, lo:hi], err_msg=f"subset {k}")


def test_done_input_state_and_temperature_vs_oracle():
    w, inp = _case(40, 6, 16, 48, 11, 5, "fp32")
    rng = np.random.default_rng(3)
    h0 = np.tanh(rng.standard_normal((40, 48))).astype(np.float32)
    c0 = rng.standard_normal((40, 48)).astype(np.float32)
    done0 = (rng.random(40) < 0.25).astype(np.uint8)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    dio = _t(done0)
    b = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=6, seed=12, tau=1.7, done=True,
                      h0=_t(h0), c0=_t(c0), done_io=dio, step0=5, traj0=100, trace=True)
    torch.cuda.synchronize()
    g = _np(b)
    ref = owm.rollout(inp["weights"], w.dims, inp["z0"], inp["mask"], T=6, seed=12, tau=1.7,
                      done_flag=True, h0=h0, c0=c0, done0=done0, step0=5, traj0=100)
    assert parity.free_run(ref, g, weights=inp["weights"], dims=w.dims, mask=inp["mask"], seed=12,
                           tau=1.7, traj=100 + np.arange(40), step0=5) <= parity.free_run_cap(40)
    parity.reanchored(w.dims, inp["weights"], inp["mask"], g, seed=12, tau=1.7, done_flag=True,
                      dtype="fp32", traj=100 + np.arange(40), step0=5, done0=done0)
    pre = done0 != 0
    assert np.all(g["actions"][:, pre] == -1) and np.all(g["dones"][:, pre] == 1)
    np.testing.assert_array_equal(g["h_T"][pre], h0[pre])
    np.testing.assert_array_equal(g["c_T"][pre], c0[pre])
    np.testing.assert_array_equal(dio.cpu().numpy(), ref["done_T"])


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_controller_step_matches_rollout_actions(dtype):
    """actions[t] of a rollout = wm_controller_step on (z_t, h_t) at step0 + t."""
    w, inp = _case(64, 5, 16, 64, 24, 3, dtype)
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    b = wmlib.rollout(m, _t(inp["z0"]), _t(inp["mask"]), T=5, seed=3, done=True, step0=2,
                      traj0=7, trace=True)
    for t in range(5):
        _, a = wmlib.controller_step(m, b.z_out[t].contiguous(), b.h_trace[t].contiguous(),
                                     _t(inp["mask"]), seed=3, step=2 + t, traj0=7,
                                     want_probs=False)
        live = b.actions[t] >= 0
        assert torch.equal(a[live], b.actions[t][live])


def test_no_done_flag_and_empty_mask_rows():
    w, inp = _case(20, 4, 8, 32, 6, 2, "fp32")
    mask = inp["mask"].copy()
    mask[[0, 7]] = 0
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    g = _np(wmlib.rollout(m, _t(inp["z0"]), _t(mask), T=4, seed=2, done=False))
    live = np.ones(20, bool)
    live[[0, 7]] = False
    assert np.all(g["dones"][:, live] == 0) and np.all(g["actions"][:, live] >= 0)
    assert np.all(g["actions"][:, ~live] == -1) and np.all(g["dones"][:, ~live] == 1)
    assert np.all(g["z_out"][:, 0] == inp["z0"][0])


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_nll_padding_ragged_and_bad_actions(dtype):
    Z, H, A, K, T, B = 24, 80, 13, 3, 9, 45
    w = wl.Workload("n", "nll", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype=dtype, seed=6)
    d = wl.make_nll_inputs(w)
    acts = d["actions"].copy()
    acts[0, :3] = [-1, A, 10 ** 6]  # outside [0, A): zero one-hot
    lengths = np.random.default_rng(1).integers(0, T + 1, size=B).astype(np.int32)
    lengths[:3] = [0, T, T + 5]
    m = wmlib.pack(d["weights"], Z, H, A, K, dtype)
    b = wmlib.nll(m, _t(d["z"]), _t(acts), _t(d["rewards"]), _t(d["dones"]), lengths=_t(lengths))
    torch.cuda.synchronize()
    ref = owm.nll(d["weights"], w.dims, d["z"], acts, d["rewards"], d["dones"], lengths=lengths,
                  dtype=dtype)
    rt = parity.RTOL[dtype]
    for k in ("loglik", "reward_se", "done_bce"):
        parity.close(getattr(b, k).cpu().numpy(), ref[k], rt, k)
    parity.close(b.means.cpu().numpy(), ref["means"], rt, "means")
    valid = np.arange(T)[:, None] < np.minimum(lengths, T)[None, :]
    assert np.all(b.loglik.cpu().numpy()[~valid] == 0)


def test_nll_all_padding_gives_zero_means():
    Z, H, A, K, T, B = 8, 16, 3, 1, 4, 6
    w = wl.Workload("n", "nll", B=B, T=T, Z=Z, H=H, A=A, K=K, dtype="fp32", seed=6)
    d = wl.make_nll_inputs(w)
    m = wmlib.pack(d["weights"], Z, H, A, K, "fp32")
    b = wmlib.nll(m, _t(d["z"]), _t(d["actions"]), _t(d["rewards"]), _t(d["dones"]),
                  lengths=_t(np.zeros(B, np.int32)))
    torch.cuda.synchronize()
    assert np.all(b.means.cpu().numpy() == 0) and np.all(b.loglik.cpu().numpy() == 0)


def test_error_paths_and_noop():
    w, inp = _case(8, 3, 8, 16, 4, 2, "fp32")
    m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = _t(inp["z0"]), _t(inp["mask"])
    with pytest.raises(wmlib.WmError):
        wmlib.rollout(m, z0, mask, T=3, seed=1, tau=0.0)
    with pytest.raises(wmlib.WmError):
        wmlib.rollout(m, z0, mask, T=3, seed=1, tau=float("inf"))
    bufs = wmlib.RolloutBuffers(m, 8, 3)
    bufs.actions.fill_(-7)
    wmlib.rollout(m, z0, mask, T=0, seed=1, bufs=bufs)  # no-op
    torch.cuda.synchronize()
    assert torch.all(bufs.actions == -7)
    with pytest.raises(wmlib.WmError):
        wmlib.pack(inp["weights"], 6, 16, 4, 2, "fp32")  # Z not a multiple of 8
