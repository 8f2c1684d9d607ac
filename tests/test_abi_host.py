"""Host-side checks of the C ABI (no GPU needed: no call here reaches a kernel)."""

import ctypes
import os
import re

import pytest

from paper_2205_01435_amd import _lib as wmlib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wm.h")

pytestmark = pytest.mark.skipif(not os.path.exists(wmlib.LIB_PATH),
                                reason="libwm.so not built (run __graft_entry__.build())")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wm_[a-z_]+)\s*\(", text)))


def test_header_declarations_are_all_exported():
    names = _declared()
    assert set(names) == set(wmlib.EXPORTS)
    lib = ctypes.CDLL(wmlib.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in wm.h but not exported"


def test_header_compiles_as_c_and_cpp(tmp_path):
    import shutil
    import subprocess
    for cc, ext in (("gcc", "c"), ("g++", "cpp")):
        if not shutil.which(cc):
            continue
        src = tmp_path / f"t.{ext}"
        src.write_text('#include "wm.h"\nint main(void){ wm_dims d = {8,16,4,2,0}; (void)d; return 0; }\n')
        subprocess.run([cc, "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), "-c", str(src),
                        "-o", str(tmp_path / f"t_{ext}.o")], check=True)


def test_version_and_sizes():
    assert "libwm" in wmlib.version()
    d = wmlib.make_dims(64, 512, 64, 5, "fp32")
    n32 = wmlib.packed_bytes(d)
    n16 = wmlib.packed_bytes(wmlib.make_dims(64, 512, 64, 5, "bf16"))
    assert n32 > 0 and n16 > 0 and n16 < n32
    # at least the canonical weights (3 matrices + controller)
    assert n32 >= 4 * (4 * 512 * (64 + 512) + 3 * 64 * 5 * 512 + 64 * (64 + 512))
    assert wmlib.workspace_bytes(d, 256, 50, 0) > 0
    assert wmlib.workspace_bytes(d, 256, 50, 1) > wmlib.workspace_bytes(d, 256, 50, 0)
    assert wmlib.workspace_bytes(d, 0, 50, 0) == 0
    # which: 0 rollout, 1 NLL, 2 controller step (no workspace), 3 training gradient
    assert wmlib.workspace_bytes(d, 256, 50, wmlib.WS_CONTROLLER) == 0
    assert wmlib.workspace_bytes(d, 256, 50, wmlib.WS_NLL_GRAD) > wmlib.workspace_bytes(d, 256, 50, 1)
    assert wmlib.workspace_bytes(d, 256, 50, 4) == 0


@pytest.mark.parametrize("dims,status", [
    ((0, 16, 4, 2), wmlib.WM_ERR_INVALID_ARG),
    ((8, 16, 4, 0), wmlib.WM_ERR_INVALID_ARG),
    ((6, 16, 4, 2), wmlib.WM_ERR_UNSUPPORTED),
    ((8, 24, 4, 2), wmlib.WM_ERR_UNSUPPORTED),
    ((8, 16, 4, 9), wmlib.WM_ERR_UNSUPPORTED),
    ((8, 16, 4096, 2), wmlib.WM_ERR_UNSUPPORTED),
])
def test_bad_dims_rejected(dims, status):
    lib = wmlib.load()
    d = wmlib.make_dims(*dims)
    assert lib.wm_packed_weights_bytes(ctypes.byref(d)) == 0
    fake = ctypes.c_void_p(256)  # never dereferenced: validation fails first
    st = lib.wm_controller_step(ctypes.byref(d), fake, 4, 0, fake, fake, fake, 1, 0, None, fake, None)
    assert st == status
    assert lib.wm_last_error().decode()


def _rollout_call(**over):
    lib = wmlib.load()
    d = wmlib.make_dims(8, 16, 4, 2)
    p = ctypes.c_void_p(4096)  # aligned dummy, never dereferenced
    args = dict(dims=ctypes.byref(d), packed=p, B=4, T=3, traj0=0, step0=0, z0=p, h0=None,
                c0=None, done_io=None, lengths=None, mask=p, seed=1, tau=1.0, flags=1, z_out=p, actions=p,
                rewards=p, dones=p, h_T=None, c_T=None, h_trace=None, c_trace=None,
                ws=p, ws_bytes=0, stream=None)
    args.update(over)
    return lib.wm_rollout(*args.values())


def test_rollout_argument_checks():
    assert _rollout_call(z0=None) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call(tau=0.0) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call(tau=float("nan")) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call(B=0) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call(T=-1) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call(flags=32) == wmlib.WM_ERR_INVALID_ARG  # an undefined flag bit
    assert _rollout_call(flags=1 << 30) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call(flags=3) == wmlib.WM_ERR_INVALID_ARG  # trace without buffers
    assert _rollout_call(z_out=ctypes.c_void_p(4100)) == wmlib.WM_ERR_INVALID_ARG  # misaligned
    assert _rollout_call(packed=ctypes.c_void_p(4112)) == wmlib.WM_ERR_INVALID_ARG
    assert _rollout_call() == wmlib.WM_ERR_WORKSPACE  # workspace too small
    # every defined flag passes the flag check (and fails later on the workspace)
    for f in (wmlib.WM_FLAG_CHECK, wmlib.WM_FLAG_STEP_MASK, wmlib.WM_FLAG_SIGMA_TAU, wmlib.WM_FLAG_TEST_ABORT):
        assert _rollout_call(flags=1 | f) == wmlib.WM_ERR_WORKSPACE, f
    assert _rollout_call(T=0) == wmlib.WM_OK  # no-op
    assert "workspace" in wmlib.load().wm_last_error().decode() or True


def test_nll_argument_checks():
    lib = wmlib.load()
    d = wmlib.make_dims(8, 16, 4, 2)
    p = ctypes.c_void_p(4096)
    st = lib.wm_nll(ctypes.byref(d), p, 4, 3, None, p, p, p, None, 0, p, p, p, None, p, 0, None)
    assert st == wmlib.WM_ERR_INVALID_ARG
    st = lib.wm_nll(ctypes.byref(d), p, 4, 3, p, p, p, p, None, 0, p, p, p, None, p, 0, None)
    assert st == wmlib.WM_ERR_WORKSPACE
    # only WM_FLAG_CHECK and WM_FLAG_TEST_ABORT are defined for the NLL pass
    st = lib.wm_nll(ctypes.byref(d), p, 4, 3, p, p, p, p, None, wmlib.WM_FLAG_DONE, p, p, p, None, p, 0, None)
    assert st == wmlib.WM_ERR_INVALID_ARG
    st = lib.wm_nll(ctypes.byref(d), p, 4, 3, p, p, p, p, None, wmlib.WM_FLAG_CHECK, p, p, p, None, p, 0, None)
    assert st == wmlib.WM_ERR_WORKSPACE


def test_workspace_status_argument_check():
    assert wmlib.load().wm_workspace_status(None, None) == wmlib.WM_ERR_INVALID_ARG


def _grad_call(dims=None, B=4, T=3, z=4096, out=4096, ws=4096, ws_bytes=0, loss=None, flags=0):
    lib = wmlib.load()
    d = dims or wmlib.make_dims(8, 16, 4, 2)
    p = ctypes.c_void_p(4096)
    zp = None if z is None else ctypes.c_void_p(z)
    o = None if out is None else ctypes.c_void_p(out)
    w = None if ws is None else ctypes.c_void_p(ws)
    return lib.wm_nll_grad(ctypes.byref(d), p, B, T, zp, p, p, p, None, flags, loss, o, p, p, p, p, p, p, p, w,
                           ws_bytes, None)


def test_nll_grad_argument_checks():
    assert _grad_call(z=None) == wmlib.WM_ERR_INVALID_ARG
    assert _grad_call(out=None) == wmlib.WM_ERR_INVALID_ARG  # every gradient output is required
    assert _grad_call(z=4100) == wmlib.WM_ERR_INVALID_ARG  # z misaligned
    assert _grad_call(B=0) == wmlib.WM_ERR_INVALID_ARG
    assert _grad_call(T=-1) == wmlib.WM_ERR_INVALID_ARG
    assert _grad_call(dims=wmlib.make_dims(8, 16, 4, 2, "bf16")) == wmlib.WM_ERR_UNSUPPORTED
    assert _grad_call(B=1 << 12, T=1 << 11) == wmlib.WM_ERR_UNSUPPORTED  # T B above 2^22
    assert _grad_call() == wmlib.WM_ERR_WORKSPACE
    assert _grad_call(T=0) == wmlib.WM_OK  # no-op
    assert _grad_call(flags=wmlib.WM_FLAG_TRACE) == wmlib.WM_ERR_INVALID_ARG


def test_nll_grad_workspace_size():
    d = wmlib.make_dims(64, 512, 64, 5, "fp32")
    nll = wmlib.workspace_bytes(d, 512, 128, wmlib.WS_NLL)
    g = wmlib.workspace_bytes(d, 512, 128, wmlib.WS_NLL_GRAD)
    # at least the NLL pass's workspace, the gate activations and their
    # gradient [T B, 4H], the c trace [T+1, B, H] and the head outputs
    assert g >= nll + 4 * (2 * 512 * 128 * 4 * 512 + 129 * 512 * 512 + 512 * 128 * (3 * 64 * 5 + 2))
    assert wmlib.workspace_bytes(d, 512, 64, wmlib.WS_NLL_GRAD) < g
    assert wmlib.workspace_bytes(wmlib.make_dims(64, 512, 64, 5, "bf16"), 512, 128, wmlib.WS_NLL_GRAD) > 0


def test_missing_library_fails_loudly(tmp_path):
    saved = wmlib._lib
    try:
        wmlib._lib = None
        with pytest.raises(wmlib.WmError):
            wmlib.load(str(tmp_path / "nope.so"))
    finally:
        wmlib._lib = saved


def test_poly_lr_matches_the_oracle_schedule():
    from oracle import train as otr
    for e in (-3, 0, 1, 1250, 2500, 4999, 5000, 7000):
        assert abs(wmlib.poly_lr(e, 3e-3, 1e-5) - otr.poly_lr(e, 3e-3, 1e-5)) <= 1e-9
    assert wmlib.poly_lr(10, 1e-3, 1e-4, epochs=20) == pytest.approx(otr.poly_lr(10, 1e-3, 1e-4, 20), rel=1e-6)
