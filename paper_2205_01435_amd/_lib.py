"""ctypes binding of libwm.so: argument marshalling only.

Every step of the hot path runs in the HIP library; this module turns torch
device tensors into pointers, allocates caller-owned buffers with torch, and
raises ``WmError`` on a non-OK status.  There is no fallback: if libwm.so is
missing or fails to load, every entry point raises.
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libwm.so")

WM_OK, WM_ERR_INVALID_ARG, WM_ERR_UNSUPPORTED, WM_ERR_WORKSPACE, WM_ERR_HIP = 0, -1, -2, -3, -4
WM_FP32, WM_BF16 = 0, 1
WM_FLAG_DONE, WM_FLAG_TRACE, WM_FLAG_CHECK, WM_FLAG_STEP_MASK, WM_FLAG_SIGMA_TAU = 1, 2, 4, 8, 16
WM_FLAG_TEST_ABORT = 0x80000000
WS_ROLLOUT, WS_NLL, WS_CONTROLLER, WS_NLL_GRAD = 0, 1, 2, 3
_DTYPES = {"fp32": WM_FP32, "bf16": WM_BF16}

# Every symbol the C header declares.
EXPORTS = ("wm_packed_weights_bytes", "wm_pack_weights", "wm_workspace_bytes", "wm_controller_step",
           "wm_rollout", "wm_rollout_noalloc", "wm_nll", "wm_nll_grad", "wm_returns", "wm_adam_step", "wm_poly_lr",
           "wm_profile_enable", "wm_profile_read", "wm_profile_reset", "wm_profile_phases",
           "wm_profile_phases_read", "wm_workspace_status",
           "wm_last_error", "wm_version")


class WmError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"libwm status {status}: {msg}")
        self.status = status


class CDims(ctypes.Structure):
    _fields_ = [("Z", ctypes.c_int32), ("H", ctypes.c_int32), ("A", ctypes.c_int32),
                ("K", ctypes.c_int32), ("dtype", ctypes.c_int32), ("N", ctypes.c_int32),
                ("L", ctypes.c_int32)]


class CWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("W_g", "b_g", "W_m", "b_m", "w_r", "b_r", "w_d", "b_d", "W_c", "b_c")]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libwm.so (once) and declare the C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise WmError(WM_ERR_UNSUPPORTED,
                      f"{path} is missing: build it with `python -m paper_2205_01435_amd.build`")
    lib = ctypes.CDLL(path)
    P, I32, U32, U64, F32, SZ = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32,
                                 ctypes.c_uint64, ctypes.c_float, ctypes.c_size_t)
    pd = ctypes.POINTER(CDims)
    lib.wm_packed_weights_bytes.argtypes = [pd]
    lib.wm_packed_weights_bytes.restype = SZ
    lib.wm_pack_weights.argtypes = [pd, ctypes.POINTER(CWeights), P, SZ, P]
    lib.wm_pack_weights.restype = I32
    lib.wm_workspace_bytes.argtypes = [pd, I32, I32, I32]
    lib.wm_workspace_bytes.restype = SZ
    lib.wm_controller_step.argtypes = [pd, P, I32, U32, P, P, P, U64, U32, P, P, P]
    lib.wm_controller_step.restype = I32
    lib.wm_rollout.argtypes = [pd, P, I32, I32, U32, U32, P, P, P, P, P, P, U64, F32, U32,
                               P, P, P, P, P, P, P, P, P, SZ, P]
    lib.wm_rollout.restype = I32
    lib.wm_rollout_noalloc.argtypes = [pd, P, I32, I32, U32, U32, P, P, P, P, P, P, U64, F32, U32,
                                       P, P, P, P, P, P, P, P, P]
    lib.wm_rollout_noalloc.restype = I32
    lib.wm_nll.argtypes = [pd, P, I32, I32, P, P, P, P, P, U32, P, P, P, P, P, SZ, P]
    lib.wm_nll.restype = I32
    lib.wm_nll_grad.argtypes = [pd, P, I32, I32, P, P, P, P, P, U32, P, P, P, P, P, P, P, P, P, P, SZ, P]
    lib.wm_nll_grad.restype = I32
    lib.wm_returns.argtypes = [I32, I32, P, P, P, F32, F32, P, P, P]
    lib.wm_returns.restype = I32
    lib.wm_adam_step.argtypes = [ctypes.c_int64, P, P, P, P, I32, F32, F32, F32, F32, P]
    lib.wm_adam_step.restype = I32
    lib.wm_poly_lr.argtypes = [I32, F32, F32, I32]
    lib.wm_poly_lr.restype = F32
    lib.wm_profile_enable.argtypes = [ctypes.c_char_p]
    lib.wm_profile_enable.restype = I32
    lib.wm_profile_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(ctypes.c_int64)]
    lib.wm_profile_read.restype = I32
    lib.wm_profile_reset.argtypes = []
    lib.wm_profile_reset.restype = I32
    lib.wm_profile_phases.argtypes = [I32]
    lib.wm_profile_phases.restype = I32
    lib.wm_profile_phases_read.argtypes = [ctypes.POINTER(ctypes.c_double), I32]
    lib.wm_profile_phases_read.restype = I32
    lib.wm_workspace_status.argtypes = [P, P]
    lib.wm_workspace_status.restype = I32
    lib.wm_last_error.argtypes = []
    lib.wm_last_error.restype = ctypes.c_char_p
    lib.wm_version.argtypes = []
    lib.wm_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int):
    if status != WM_OK:
        raise WmError(status, load().wm_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dev_f32(x, device):
    return torch.as_tensor(x, dtype=torch.float32).to(device).contiguous()


def _need(name, t, dtype, shape, device=None, optional=False):
    """Checks a tensor argument before its pointer crosses the C ABI."""
    if t is None:
        if optional:
            return
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the model on {device}")


def _mask_dtype(t):
    return t.dtype if t is not None and t.dtype in (torch.uint8, torch.bool) else torch.uint8


def status(bufs) -> None:
    """Wait for the current stream and raise WmError if the last call that
    used ``bufs.workspace`` failed on the device (a timed-out barrier wait of
    the persistent kernels, or WM_FLAG_CHECK violations)."""
    _check(load().wm_workspace_status(_ptr(bufs.workspace), _stream()))


@dataclass
class Model:
    """Packed weights on a device plus their dims."""

    dims: CDims
    packed: torch.Tensor
    Z: int
    H: int
    A: int
    K: int
    dtype: str


def make_dims(Z, H, A, K, dtype="fp32", N=0, L=0) -> CDims:
    """N, L > 0: the two-level controller (N xfers + NO-OP, L locations, A = N L)."""
    return CDims(Z, H, A, K, _DTYPES[dtype], N, L)


def packed_bytes(dims: CDims) -> int:
    return load().wm_packed_weights_bytes(ctypes.byref(dims))


def workspace_bytes(dims: CDims, B: int, T: int, which: int) -> int:
    return load().wm_workspace_bytes(ctypes.byref(dims), B, T, which)


def pack(weights: dict, Z: int, H: int, A: int, K: int, dtype: str = "fp32",
         device="cuda", N: int = 0, L: int = 0) -> Model:
    """Copy canonical float32 weights to the device and pack them (N, L > 0:
    the two-level controller, W_c [N+1+L, Z+H])."""
    lib = load()
    dims = make_dims(Z, H, A, K, dtype, N, L)
    n = lib.wm_packed_weights_bytes(ctypes.byref(dims))
    if n == 0:
        raise WmError(WM_ERR_UNSUPPORTED, lib.wm_last_error().decode())
    canon = {k: _dev_f32(np_or_t, device).reshape(-1) for k, np_or_t in weights.items()}
    packed = torch.empty(n, dtype=torch.uint8, device=device)
    cw = CWeights(*[ctypes.c_void_p(canon[k].data_ptr()) for k in
                    ("W_g", "b_g", "W_m", "b_m", "w_r", "b_r", "w_d", "b_d", "W_c", "b_c")])
    _check(lib.wm_pack_weights(ctypes.byref(dims), ctypes.byref(cw), _ptr(packed), n, _stream()))
    torch.cuda.current_stream().synchronize()  # canon tensors may be freed after return
    return Model(dims, packed, Z, H, A, K, dtype)


def repack(m: Model, canon: dict):
    """Re-pack canonical float32 device tensors (every weight, the
    controller's included) into m.packed on the current stream (after an
    optimiser step); nothing is allocated and nothing waits."""
    lib = load()
    for k in ("W_g", "b_g", "W_m", "b_m", "w_r", "b_r", "w_d", "b_d", "W_c", "b_c"):
        t = canon[k]
        assert t.is_cuda and t.dtype == torch.float32 and t.is_contiguous(), k
    cw = CWeights(*[ctypes.c_void_p(canon[k].data_ptr()) for k in
                    ("W_g", "b_g", "W_m", "b_m", "w_r", "b_r", "w_d", "b_d", "W_c", "b_c")])
    _check(lib.wm_pack_weights(ctypes.byref(m.dims), ctypes.byref(cw), _ptr(m.packed), m.packed.numel(),
                               _stream()))


def two_level_mask(m: Model, xm, lm):
    """The one buffer the library reads for the two-level controller: the
    xfer masks [B, N+1], then the location masks [B, N, L] (uint8)."""
    return _two_level_mask(m, (xm, lm), xm.shape[0])


def _two_level_mask(m: Model, mask, B: int):
    """(xfer mask [B, N+1], location mask [B, N, L]) as the one buffer the
    library reads, xfer masks first; a flat buffer of that layout is taken
    as it is."""
    N, L = m.dims.N, m.dims.L
    dev = m.packed.device
    if isinstance(mask, torch.Tensor):
        _need("two-level mask", mask, _mask_dtype(mask), (B * (N + 1) + B * N * L,), dev)
        return mask
    xm, lm = mask
    _need("xfer mask", xm, _mask_dtype(xm), (B, N + 1), dev)
    _need("location mask", lm, _mask_dtype(lm), (B, N, L), dev)
    return torch.cat([xm.reshape(-1), lm.reshape(-1)]).contiguous()


def controller_step(m: Model, z, h, mask, seed: int, step: int, traj0: int = 0,
                    want_probs: bool = True):
    """Returns (probs or None, action [B] int32).  One-level: probs [B, A].
    Two-level (N > 0): ``mask`` is (xfer mask [B, N+1], location mask
    [B, N, L]) and probs [B, N+1+L] (always returned)."""
    lib = load()
    B = z.shape[0]
    dev = m.packed.device
    _need("z", z, torch.float32, (B, m.Z), dev)
    _need("h", h, torch.float32, (B, m.H), dev)
    if m.dims.N > 0:
        mask = _two_level_mask(m, mask, B)
        probs = torch.empty((B, m.dims.N + 1 + m.dims.L), dtype=torch.float32, device=dev)
    else:
        _need("mask", mask, _mask_dtype(mask), (B, m.A), dev)
        probs = torch.empty((B, m.A), dtype=torch.float32, device=dev) if want_probs else None
    action = torch.empty(B, dtype=torch.int32, device=dev)
    _check(lib.wm_controller_step(ctypes.byref(m.dims), _ptr(m.packed), B, traj0, _ptr(z),
                                  _ptr(h), _ptr(mask), seed, step, _ptr(probs), _ptr(action),
                                  _stream()))
    return probs, action


class RolloutBuffers:
    """Caller-owned device buffers of one rollout shape (reusable across calls)."""

    def __init__(self, m: Model, B: int, T: int, trace: bool = False, final_state: bool = True,
                 workspace: bool = True):
        dev = m.packed.device
        self.B, self.T, self.Z, self.H = B, T, m.Z, m.H
        self.z_out = torch.empty((T + 1, B, m.Z), dtype=torch.float32, device=dev)
        self.actions = torch.empty((T, B), dtype=torch.int32, device=dev)
        self.rewards = torch.empty((T, B), dtype=torch.float32, device=dev)
        self.dones = torch.empty((T, B), dtype=torch.uint8, device=dev)
        self.h_T = torch.empty((B, m.H), dtype=torch.float32, device=dev) if final_state else None
        self.c_T = torch.empty((B, m.H), dtype=torch.float32, device=dev) if final_state else None
        self.h_trace = (torch.empty((T + 1, B, m.H), dtype=torch.float32, device=dev)
                        if trace else None)
        self.c_trace = (torch.empty((T + 1, B, m.H), dtype=torch.float32, device=dev)
                        if trace else None)
        nws = workspace_bytes(m.dims, B, T, WS_ROLLOUT) if workspace else 0
        self.workspace = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev) if workspace else None
        self.ws_bytes = nws


def rollout(m: Model, z0, mask, *, T: int, seed: int, tau: float = 1.0, done: bool = True,
            traj0: int = 0, step0: int = 0, h0=None, c0=None, done_io=None, lengths=None,
            trace: bool = False,
            bufs: RolloutBuffers | None = None, sigma_tau: bool = False, check: bool = False,
            extra_flags: int = 0, noalloc: bool = False) -> RolloutBuffers:
    """Launch wm_rollout on the current stream; returns the filled buffers
    (``lengths`` [B] int32: per-trajectory horizons, later steps padded;
    ``sigma_tau`` sets WM_FLAG_SIGMA_TAU; a [T, B, A] mask sets
    WM_FLAG_STEP_MASK; ``check`` sets WM_FLAG_CHECK, which waits for the
    stream; ``noalloc`` calls wm_rollout_noalloc, whose workspace is the
    library's static device scratch)."""
    lib = load()
    B = z0.shape[0]
    dev = m.packed.device
    _need("z0", z0, torch.float32, (B, m.Z), dev)
    _need("h0", h0, torch.float32, (B, m.H), dev, optional=True)
    _need("c0", c0, torch.float32, (B, m.H), dev, optional=True)
    _need("done_io", done_io, _mask_dtype(done_io), (B,), dev, optional=True)
    _need("lengths", lengths, torch.int32, (B,), dev, optional=True)
    if m.dims.N > 0:
        mask = _two_level_mask(m, mask, B)
        step_mask = False
    else:
        step_mask = mask is not None and mask.dim() == 3
        want = (T, B, m.dims.A) if step_mask else (B, m.dims.A)
        _need("mask", mask, _mask_dtype(mask), want, dev)
    if bufs is None:
        bufs = RolloutBuffers(m, B, T, trace=trace, workspace=not noalloc)
    if T > 0 and ((bufs.B, bufs.T) != (B, T) or bufs.Z != m.Z or bufs.H != m.H):
        raise ValueError(f"buffers for B={bufs.B} T={bufs.T} Z={bufs.Z} H={bufs.H}; the call has "
                         f"B={B} T={T} Z={m.Z} H={m.H}")
    if trace and bufs.h_trace is None:
        raise ValueError("trace=True needs buffers made with trace=True")
    flags = (WM_FLAG_DONE if done else 0) | (WM_FLAG_TRACE if trace else 0) | \
        (WM_FLAG_SIGMA_TAU if sigma_tau else 0) | (WM_FLAG_STEP_MASK if step_mask else 0) | \
        (WM_FLAG_CHECK if check else 0) | extra_flags
    common = (ctypes.byref(m.dims), _ptr(m.packed), B, T, traj0, step0, _ptr(z0), _ptr(h0), _ptr(c0),
              _ptr(done_io), _ptr(lengths), _ptr(mask), seed, tau, flags, _ptr(bufs.z_out), _ptr(bufs.actions),
              _ptr(bufs.rewards), _ptr(bufs.dones), _ptr(bufs.h_T), _ptr(bufs.c_T),
              _ptr(bufs.h_trace if trace else None), _ptr(bufs.c_trace if trace else None))
    if noalloc:
        _check(lib.wm_rollout_noalloc(*common, _stream()))
    else:
        if bufs.workspace is None:
            raise ValueError("these buffers have no workspace (made for wm_rollout_noalloc)")
        _check(lib.wm_rollout(*common, _ptr(bufs.workspace), bufs.ws_bytes, _stream()))
    return bufs


class NllBuffers:
    def __init__(self, m: Model, B: int, T: int):
        dev = m.packed.device
        self.B, self.T = B, T
        self.loglik = torch.empty((T, B), dtype=torch.float32, device=dev)
        self.reward_se = torch.empty((T, B), dtype=torch.float32, device=dev)
        self.done_bce = torch.empty((T, B), dtype=torch.float32, device=dev)
        self.means = torch.empty(3, dtype=torch.float32, device=dev)
        nws = workspace_bytes(m.dims, B, T, WS_NLL)
        self.workspace = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
        self.ws_bytes = nws


def _nll_inputs(m: Model, z, actions, rewards, dones, lengths):
    T, B = actions.shape
    dev = m.packed.device
    _need("actions", actions, torch.int32, (T, B), dev)
    _need("z", z, torch.float32, (T + 1, B, m.Z), dev)
    _need("rewards", rewards, torch.float32, (T, B), dev)
    _need("dones", dones, _mask_dtype(dones), (T, B), dev)
    _need("lengths", lengths, torch.int32, (B,), dev, optional=True)
    return T, B


def nll(m: Model, z, actions, rewards, dones, lengths=None,
        bufs: NllBuffers | None = None, check: bool = False, extra_flags: int = 0) -> NllBuffers:
    """Launch wm_nll on the current stream; returns the filled buffers
    (``check`` sets WM_FLAG_CHECK, which waits for the stream)."""
    lib = load()
    T, B = _nll_inputs(m, z, actions, rewards, dones, lengths)
    if bufs is None:
        bufs = NllBuffers(m, B, T)
    if (bufs.B, bufs.T) != (B, T):
        raise ValueError(f"buffers for B={bufs.B} T={bufs.T}; the call has B={B} T={T}")
    flags = (WM_FLAG_CHECK if check else 0) | extra_flags
    _check(lib.wm_nll(ctypes.byref(m.dims), _ptr(m.packed), B, T, _ptr(z), _ptr(actions),
                      _ptr(rewards), _ptr(dones), _ptr(lengths), flags, _ptr(bufs.loglik),
                      _ptr(bufs.reward_se), _ptr(bufs.done_bce), _ptr(bufs.means),
                      _ptr(bufs.workspace), bufs.ws_bytes, _stream()))
    return bufs


GRAD_SHAPES = {  # canonical gradient shapes, as the weights
    "W_g": lambda Z, H, A, K: (4 * H, Z + A + H), "b_g": lambda Z, H, A, K: (4 * H,),
    "W_m": lambda Z, H, A, K: (3 * Z * K, H), "b_m": lambda Z, H, A, K: (3 * Z * K,),
    "w_r": lambda Z, H, A, K: (H,), "b_r": lambda Z, H, A, K: (1,),
    "w_d": lambda Z, H, A, K: (H,), "b_d": lambda Z, H, A, K: (1,),
}


def flat_views(flat, Z: int, H: int, A: int, K: int) -> dict:
    """Views of a flat float32 tensor as the world-model weights, in the
    order of GRAD_SHAPES (the layout of GradBuffers.flat)."""
    out, o = {}, 0
    for k, f in GRAD_SHAPES.items():
        shp = f(Z, H, A, K)
        n = math.prod(shp)
        out[k] = flat[o:o + n].view(shp)
        o += n
    return out


class GradBuffers:
    """Loss, gradients (views of one flat buffer, GRAD_SHAPES order) and the
    workspace of one wm_nll_grad shape."""

    def __init__(self, m: Model, B: int, T: int):
        dev = m.packed.device
        self.B, self.T = B, T
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        n = sum(math.prod(f(m.Z, m.H, m.A, m.K)) for f in GRAD_SHAPES.values())
        self.flat = torch.empty(n, dtype=torch.float32, device=dev)
        self.grads = flat_views(self.flat, m.Z, m.H, m.A, m.K)
        nws = workspace_bytes(m.dims, B, T, WS_NLL_GRAD)
        self.workspace = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
        self.ws_bytes = nws


def nll_grad(m: Model, z, actions, rewards, dones, lengths=None,
             bufs: GradBuffers | None = None, check: bool = False, extra_flags: int = 0) -> GradBuffers:
    """Launch wm_nll_grad on the current stream: the training loss (summed
    NLL means) and its gradient in the canonical weight layout."""
    lib = load()
    T, B = _nll_inputs(m, z, actions, rewards, dones, lengths)
    if bufs is None:
        bufs = GradBuffers(m, B, T)
    if (bufs.B, bufs.T) != (B, T):
        raise ValueError(f"buffers for B={bufs.B} T={bufs.T}; the call has B={B} T={T}")
    g = bufs.grads
    flags = (WM_FLAG_CHECK if check else 0) | extra_flags
    _check(lib.wm_nll_grad(ctypes.byref(m.dims), _ptr(m.packed), B, T, _ptr(z), _ptr(actions),
                           _ptr(rewards), _ptr(dones), _ptr(lengths), flags, _ptr(bufs.loss),
                           _ptr(g["W_g"]), _ptr(g["b_g"]), _ptr(g["W_m"]), _ptr(g["b_m"]),
                           _ptr(g["w_r"]), _ptr(g["b_r"]), _ptr(g["w_d"]), _ptr(g["b_d"]),
                           _ptr(bufs.workspace), bufs.ws_bytes, _stream()))
    return bufs


def returns(rewards, dones, gamma: float, values=None, lam: float = 1.0, out=None, adv=None):
    """Launch wm_returns on the current stream over device tensors
    rewards [T, B] float32 and dones [T, B] uint8 (values [T+1, B] float32 or
    None).  Returns (returns [T, B], advantages [T, B] or None)."""
    lib = load()
    T, B = rewards.shape
    if out is None:
        out = torch.empty((T, B), dtype=torch.float32, device=rewards.device)
    if values is not None and adv is None:
        adv = torch.empty((T, B), dtype=torch.float32, device=rewards.device)
    _check(lib.wm_returns(B, T, _ptr(rewards), _ptr(dones), _ptr(values), gamma, lam, _ptr(out),
                          _ptr(adv if values is not None else None), _stream()))
    return out, (adv if values is not None else None)


def adam_step(params, grads, m, v, step: int, lr: float, beta1: float = 0.9, beta2: float = 0.999,
              eps: float = 1e-8):
    """Launch wm_adam_step on the current stream over flat float32 device
    tensors of one size (updated in place)."""
    n = params.numel()
    assert grads.numel() == n and m.numel() == n and v.numel() == n
    _check(load().wm_adam_step(n, _ptr(params), _ptr(grads), _ptr(m), _ptr(v), step, lr, beta1, beta2,
                               eps, _stream()))


def poly_lr(epoch: int, lr0: float, lr_end: float, epochs: int = 5000) -> float:
    return float(load().wm_poly_lr(epoch, lr0, lr_end, epochs))


def profile_enable(prefix: str | None):
    """Bracket launches of kernels whose name starts with ``prefix`` with HIP
    events (None turns it off)."""
    _check(load().wm_profile_enable(None if prefix is None else prefix.encode()))


def profile_read(prefix: str | None = None) -> tuple[float, int]:
    """(summed milliseconds, launch count) of the recorded launches."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(load().wm_profile_read(None if prefix is None else prefix.encode(), ctypes.byref(ms),
                                  ctypes.byref(n)))
    return ms.value, n.value


def profile_reset():
    _check(load().wm_profile_reset())


PHASE_SLOTS = ("T", "step", "ctrl", "ctrl_barrier", "gates", "gates_barrier", "mdn", "mdn_barrier",
               "ctrl_mean", "gates_mean", "mdn_mean", "setup", "tail")


def profile_phases(on: bool):
    """Stamp the phase boundaries of later persistent-kernel launches."""
    _check(load().wm_profile_phases(1 if on else 0))


def profile_phases_read() -> dict:
    """Per-step phase durations (us) of the last stamped launch, by slot."""
    out = (ctypes.c_double * len(PHASE_SLOTS))()
    _check(load().wm_profile_phases_read(out, len(PHASE_SLOTS)))
    return dict(zip(PHASE_SLOTS, list(out)))


def version() -> str:
    return load().wm_version().decode()
