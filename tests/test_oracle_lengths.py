"""Pins of the oracle's variable-length rollouts (section 3.3.1: sequences of
different lengths are zero-padded and masked).

* lengths = T everywhere is the plain rollout, bit for bit;
* a trajectory with horizon L agrees with the plain rollout on its first L
  steps, as the random streams are keyed by step and trajectory and rows do
  not interact (discrete outputs exactly; floats to 1e-12, since numpy's
  products over a different set of live rows round differently); its final
  state is the plain rollout's state after L steps (or the state it froze
  in); every step from L on is padding: action -1, reward 0, done 0,
  z_out 0;
* horizon 0 leaves the initial state and pads every step;
* a horizon beyond T is clamped to T;
* the done flag returned is the trajectory's own (padding is not an end).
"""

import numpy as np

from oracle import wm as owm
from paper_2205_01435_amd import workloads as wl


def _case(dtype="fp32"):
    w = wl.Workload("len", "rollout", B=9, T=7, Z=8, H=16, A=6, K=3, dtype=dtype, seed=23)
    return w, wl.make_rollout_inputs(w)


def _run(w, inp, **kw):
    return owm.rollout(inp["weights"], w.dims, inp["z0"], inp["mask"], T=w.T, seed=5, tau=1.2,
                       done_flag=True, dtype=w.dtype, **kw)


def test_full_lengths_are_the_plain_rollout():
    w, inp = _case()
    a = _run(w, inp)
    b = _run(w, inp, lengths=np.full(w.B, w.T))
    for k in ("z_out", "actions", "rewards", "dones", "h_T", "c_T", "done_T", "h_trace"):
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)  # the same rows in every product


def test_prefix_state_and_padding():
    for dtype in ("fp32", "bf16"):
        w, inp = _case(dtype)
        full = _run(w, inp)
        lens = np.array([0, 1, 3, 7, 2, 5, 9, 4, 6])  # 9 > T: clamped
        r = _run(w, inp, lengths=lens)
        for b, L in enumerate(np.minimum(lens, w.T)):
            np.testing.assert_array_equal(r["actions"][:L, b], full["actions"][:L, b])
            np.testing.assert_array_equal(r["dones"][:L, b], full["dones"][:L, b])
            close = dict(rtol=1e-12, atol=1e-14)
            np.testing.assert_allclose(r["rewards"][:L, b], full["rewards"][:L, b], **close)
            np.testing.assert_allclose(r["z_out"][:L + 1, b], full["z_out"][:L + 1, b], **close)
            # the final state is the state after step L - 1
            np.testing.assert_allclose(r["h_T"][b], full["h_trace"][L, b], **close)
            np.testing.assert_allclose(r["c_T"][b], full["c_trace"][L, b], **close)
            assert r["done_T"][b] == (full["dones"][:L, b].any() if L else 0)
            # padding
            assert np.all(r["actions"][L:, b] == -1)
            assert np.all(r["rewards"][L:, b] == 0) and np.all(r["dones"][L:, b] == 0)
            assert np.all(r["z_out"][L + 1:, b] == 0)
            assert np.all(np.isnan(r["action_margin"][L:, b]))


def test_zero_length_keeps_the_initial_state():
    w, inp = _case()
    rng = np.random.default_rng(1)
    h0 = np.tanh(rng.standard_normal((w.B, w.H)))
    c0 = rng.standard_normal((w.B, w.H))
    r = _run(w, inp, lengths=np.zeros(w.B, np.int64), h0=h0, c0=c0)
    np.testing.assert_array_equal(r["z_out"][0], inp["z0"])
    assert np.all(r["z_out"][1:] == 0) and np.all(r["actions"] == -1) and np.all(r["dones"] == 0)
    np.testing.assert_array_equal(r["h_T"], h0)
    np.testing.assert_array_equal(r["c_T"], c0)
    assert np.all(r["done_T"] == 0)
