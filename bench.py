#!/usr/bin/env python3
"""Throughput of the World-Model dream hot path on one MI355X.

One step = one dream rollout of the xlarge workload, the largest of the five
(B = 16384 trajectories x T = 64 steps, Z = 128, H = 1024, A = 256, K = 8,
bf16 weights and GEMM operands, fp32 accumulate and mixture arithmetic, done
head on, mask p = 0.1): per step the controller with its masked Gumbel-max
action, the LSTM gates and cell, the mixture head with its component pick
and Box-Muller draw, the reward and done heads, freeze/commit.
value = B * T / seconds per step (imagined transitions/s).  Inputs are
resident in HBM before the timed region; weights are packed once, outside
it.  The teacher-forced NLL pass is measured on its own workload (B 512,
T 128, fp32) in the per-workload table, as are the other four workloads.

Prints ONE JSON line (rank 0, N = 1).  --gpus above 1 exits with a message:
the benchmark measures one GPU.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "imagined transitions/sec (B×T) + MDN-NLL tokens/sec; % of MFMA/HBM peak"
PEAK = {"fp32": 157.3e12, "bf16": 2516.6e12}  # dense MFMA, FLOP/s
HBM_PEAK = 8.0e12  # B/s
HEADLINE = "xlarge_rollout"
CPU_ROWS = 512  # trajectories of the oracle's timed sample


def flops_per_transition(w) -> float:
    """Algorithmic flops of one dream transition (the one-hot product is a
    column gather and is not counted)."""
    Z, H, A, K = w.Z, w.H, w.A, w.K
    return 2.0 * (4 * H * (Z + H) + 3 * Z * K * H + A * (Z + H) + 2 * H)


def flops_per_token(w) -> float:
    Z, H, K = w.Z, w.H, w.K
    return 2.0 * (4 * H * (Z + H) + 3 * Z * K * H + 2 * H)


def kernel_flops_per_launch(name: str, w, B: int, T: int) -> float:
    """Algorithmic flops of one launch of a kernel class of a dream rollout.
    persist: the whole rollout (every phase of every step, one launch);
    gates / mdn / ctrl: one dream step of the multi-launch path (the gate
    GEMM; the mixture head with the reward and done columns counted in the
    controller, which computes them; the controller's logits)."""
    Z, H, A, K = w.Z, w.H, w.A, w.K
    if name == "persist":
        return B * T * flops_per_transition(w)
    if name == "gates":
        return 2.0 * B * 4 * H * (Z + H)
    if name == "mdn":
        return 2.0 * B * 3 * Z * K * H
    if name == "ctrl":
        return 2.0 * B * (A * (Z + H) + 2 * H)
    return 0.0


def weight_stream_bytes_per_step(w) -> float:
    """Bytes of weights a step must move if nothing stays on chip (all
    matrices at their precision + fp32 biases + min(B, A) gathered columns)."""
    esz = 4 if w.dtype == "fp32" else 2
    Z, H, A, K = w.Z, w.H, w.A, w.K
    mats = 4 * H * (Z + H) + 3 * Z * K * H + 2 * H + A * (Z + H)
    gathered = min(w.B, A) * 4 * H
    biases = 4 * H + 3 * Z * K + 2 + A
    return mats * esz + gathered * esz + biases * 4


def _range(torch, name):
    """A roctx range around a region (visible to rocprofv3 --marker-trace)."""
    try:
        torch.cuda.nvtx.range_push(name)
        return lambda: torch.cuda.nvtx.range_pop()
    except Exception:  # noqa: BLE001
        return lambda: None


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing")
    ap.add_argument("--no-workloads", action="store_true", help="skip the per-workload table")
    ap.add_argument("--rows", default="", help="comma-separated rows of the per-workload table to run "
                    "(default: all)")
    ap.add_argument("--cpu-seconds", type=float, default=20.0, help="oracle sample budget")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} (WORLD_SIZE {world}) is not "
              "supported: the rollout shards by trajectory with no exchange, so N GPUs run N "
              "independent copies of this benchmark.", file=sys.stderr)
        return 2

    import torch

    from paper_2205_01435_amd import _lib as wmlib
    from paper_2205_01435_amd import workloads as wl
    from paper_2205_01435_amd.traffic import read_summary

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wmlib.load()
    dev = torch.device("cuda:0")

    def cuda(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    w = wl.WORKLOADS[HEADLINE]
    B, T = w.B, w.T
    roll_in = wl.make_rollout_inputs(w)
    model = wmlib.pack(roll_in["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = cuda(roll_in["z0"]), cuda(roll_in["mask"])
    rbufs = wmlib.RolloutBuffers(model, B, T, trace=False)

    def step(i):
        wmlib.rollout(model, z0, mask, T=T, seed=w.seed + i, tau=w.tau, done=w.done, bufs=rbufs)

    # warmup, with every kernel class timed to find the dominant one
    classes = ["persist", "ctrl", "gates", "mdn", "init", "finish"]
    wmlib.profile_reset()
    wmlib.profile_enable("")
    nwarm = max(args.warmup, 1)
    for i in range(nwarm):
        step(i)
    torch.cuda.synchronize()
    warm = {c: wmlib.profile_read(c) for c in classes}
    dominant = max(classes, key=lambda c: warm[c][0])
    wmlib.profile_enable(None)
    wmlib.profile_reset()

    # timed region: K steps; each launch of the dominant kernel carries a
    # start/stop event pair stamped by its own dispatch (on the stream it runs
    # on, the current torch stream)
    def timed(prefix):
        wmlib.profile_reset()
        wmlib.profile_enable(prefix)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        done = _range(torch, "timed_steps" if prefix is None else "instrumented_steps")
        t0 = time.perf_counter()
        ev0.record()
        for i in range(args.steps):
            step(args.warmup + i)
        ev1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        done()
        kern = wmlib.profile_read(prefix) if prefix is not None else (0.0, 0)
        wmlib.profile_enable(None)
        wmlib.profile_reset()
        return ev0.elapsed_time(ev1), wall, kern

    # value: K steps with nothing but the two bracketing events; roofline: the
    # same K steps again with dispatch-stamped events on the dominant kernel
    # (they add host work per launch, so they stay out of the throughput)
    ms_total, t_wall, _ = timed(None)
    ms_inst, _, (k_ms, k_n) = timed(dominant)
    ms_step = ms_total / args.steps
    value = B * T / (ms_step / 1e3)
    live = int((rbufs.actions >= 0).sum().item())

    avg_ms = k_ms / max(k_n, 1)
    flops_launch = kernel_flops_per_launch(dominant, w, B, T)
    achieved = flops_launch / (avg_ms / 1e3) if avg_ms > 0 else 0.0
    traffic = read_summary(os.path.join(ROOT, "profiles", f"traffic_{dominant}_{HEADLINE}_bf16.md"))
    roofline = {"kernel": dominant, "bound": "mfma", "achieved": achieved / 1e12,
                "peak": PEAK[w.dtype] / 1e12, "unit": "TFLOP/s",
                "frac": achieved / PEAK[w.dtype], "traffic": traffic,
                "traffic_unit": "bytes per launch (HBM, rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
                "avg_launch_us": avg_ms * 1e3, "launches": k_n,
                "measured": "dispatch-stamped HIP events on every launch of the kernel over a "
                            "second pass of the same K steps, on the launch stream",
                "flops_per_launch": flops_launch}

    per_step_kernel_ms = {c: warm[c][0] / nwarm for c in classes if warm[c][1]}
    out = {
        "metric": METRIC, "value": value, "unit": "transitions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; Xavier-uniform weights, N(0,1) latents, Bernoulli(0.1) masks)",
        "config": {"workload": f"{HEADLINE}: dream rollout B={B} T={T} Z={w.Z} H={w.H} A={w.A} K={w.K} "
                               "bf16 (fp32 accumulate and mixture math), done head on, mask p 0.1",
                   "B": B, "T": T, "Z": w.Z, "H": w.H, "A": w.A, "K": w.K, "tau": w.tau},
        "breakdown": {"rollout_tflops": B * T * flops_per_transition(w) / (ms_step / 1e3) / 1e12,
                      "rollout_frac_bf16_peak": B * T * flops_per_transition(w) / (ms_step / 1e3)
                      / PEAK[w.dtype],
                      "live_transitions_last_rollout": live,
                      "kernel_ms_per_rollout_warmup": {c: round(v, 4) for c, v in per_step_kernel_ms.items()},
                      "launches_per_rollout": {c: warm[c][1] // nwarm for c in classes if warm[c][1]},
                      "wall_s_timed_region": t_wall,
                      "ms_per_step_with_kernel_events": ms_inst / args.steps},
        "roofline": roofline,
    }

    if not args.no_workloads:
        out["workloads"] = workload_table(wmlib, wl, torch, cuda, {r for r in args.rows.split(",") if r})
        nll = out["workloads"].get("nll")
        if nll:
            out["nll"] = {"metric": "MDN-NLL tokens/sec", "value": nll["per_s"], "unit": "tokens/s",
                          "ms": nll["ms"], "config": "nll: teacher-forced NLL pass B=512 T=128 Z=64 H=512 "
                          "A=64 K=5 fp32", "frac_mfma_peak": nll["frac_mfma_peak"]}

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, roll_in, args.cpu_seconds)

    print(json.dumps(out), flush=True)
    return 0


def _median_ms(torch, fn, min_reps: int = 10, min_total_s: float = 1.0, max_reps: int = 2000) -> tuple:
    """3 warm-up calls, then the median of per-call event timings over at
    least ``min_reps`` calls and at least ``min_total_s`` seconds."""
    for i in range(3):
        fn(i)
    torch.cuda.synchronize()
    times = []
    i = 3
    t_start = time.perf_counter()
    while len(times) < min_reps or (sum(times) < min_total_s * 1e3 and len(times) < max_reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn(i)
        b.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(b))
        i += 1
        if time.perf_counter() - t_start > 20.0 and len(times) >= min_reps:
            break
    return float(np.median(times)), len(times)


def workload_table(wmlib, wl, torch, cuda, only=frozenset()) -> dict:
    """Whole-call timing of every workload (median of at least 10 calls and
    1 s after 3 warm-ups); `only` (non-empty) restricts the table to the rows
    it names."""
    res = {}
    for name, w in wl.WORKLOADS.items():
        if only and name not in only:
            continue
        if w.kind == "rollout":
            inp = wl.make_rollout_inputs(w)
            m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
            z0, mask = cuda(inp["z0"]), cuda(inp["mask"])
            bufs = wmlib.RolloutBuffers(m, w.B, w.T)
            fn = lambda i: wmlib.rollout(m, z0, mask, T=w.T, seed=w.seed + i, tau=w.tau,  # noqa: E731
                                         done=w.done, bufs=bufs)
            fl = flops_per_transition(w)
        else:
            d = wl.make_nll_inputs(w)
            m = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, w.dtype)
            args = [cuda(d[k]) for k in ("z", "actions", "rewards", "dones")]
            bufs = wmlib.NllBuffers(m, w.B, w.T)
            fn = lambda i: wmlib.nll(m, *args, bufs=bufs)  # noqa: E731
            fl = flops_per_token(w)
        ms, reps = _median_ms(torch, fn)
        n = w.B * w.T
        row = {"ms": ms, "reps": reps, "per_s": n / (ms / 1e3),
               "unit": "transitions/s" if w.kind == "rollout" else "tokens/s",
               "tflops": n * fl / (ms / 1e3) / 1e12, "frac_mfma_peak": n * fl / (ms / 1e3) / PEAK[w.dtype]}
        if name == "tiny_rollout":
            gb = weight_stream_bytes_per_step(w) * w.T
            row["weight_stream_GBps"] = gb / (ms / 1e3) / 1e9
            row["frac_hbm_peak"] = gb / (ms / 1e3) / HBM_PEAK
        res[name] = row
        del bufs, m
        torch.cuda.empty_cache()
    extra = {"returns_gae_xlarge": lambda: returns_row(wmlib, torch, cuda),
             "two_level_rollout_n288": lambda: two_level_row(wmlib, wl, torch, cuda, 288),
             "two_level_rollout_n80": lambda: two_level_row(wmlib, wl, torch, cuda, 80),
             "adam_xlarge_wm": lambda: adam_row(wmlib, torch),
             "library_gemm_xlarge": lambda: library_gemm_row(torch),
             "train_step_nll": lambda: train_step_row(wmlib, wl, torch, cuda)}
    for name, fn in extra.items():
        if not only or name in only:
            res[name] = fn()
    return res


def train_step_row(wmlib, wl, torch, cuda) -> dict:
    """One world-model training step on the NLL workload (B 512 sequences,
    T 128, Z 64, H 512, A 64, K 5, fp32): the loss gradient by
    backpropagation through time (wm_nll_grad), Adam on the flat canonical
    parameters (wm_adam_step) and the re-pack for the next forward pass.
    Algorithmic FLOPs per token: three times the forward products, 2 4H (Z+H)
    for the gates and 2 H (3ZK+2) for the heads (the forward, the gradient
    with respect to the inputs, the gradient with respect to the weights)."""
    w = wl.WORKLOADS["nll"]
    d = wl.make_nll_inputs(w)
    m = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, "fp32")
    args = [cuda(d[k]) for k in ("z", "actions", "rewards", "dones")]
    gb = wmlib.GradBuffers(m, w.B, w.T)
    params = torch.cat([cuda(np.asarray(d["weights"][k], np.float32).reshape(-1))
                        for k in wmlib.GRAD_SHAPES])
    canon = wmlib.flat_views(params, w.Z, w.H, w.A, w.K)
    canon["W_c"] = cuda(np.asarray(d["weights"]["W_c"], np.float32))
    canon["b_c"] = cuda(np.asarray(d["weights"]["b_c"], np.float32))
    mom, vel = torch.zeros_like(params), torch.zeros_like(params)

    def step(i):
        wmlib.nll_grad(m, *args, bufs=gb)
        wmlib.adam_step(params, gb.flat, mom, vel, i + 1, 1e-4)
        wmlib.repack(m, canon)

    ms, reps = _median_ms(torch, step)
    wmlib.profile_reset()
    wmlib.profile_enable("")
    step(reps + 3)
    torch.cuda.synchronize()
    parts = {p: wmlib.profile_read(p)[0] for p in ("nll_persist", "mdn", "grad_gemm_bptt", "grad_gemm",
                                                  "grad_lstm", "grad_", "adam", "pack")}
    wmlib.profile_enable(None)
    wmlib.profile_reset()
    parts["grad_gemm"] -= parts["grad_gemm_bptt"]
    parts["grad_other"] = parts.pop("grad_") - parts["grad_gemm"] - parts["grad_gemm_bptt"] - parts["grad_lstm"]
    fwd = 2 * 4 * w.H * (w.Z + w.H) + 2 * w.H * (3 * w.Z * w.K + 2)
    n = w.B * w.T
    fl = 3.0 * fwd * n
    return {"ms": ms, "reps": reps, "tokens_per_s": n / (ms / 1e3), "flops_per_step": fl, "tflops": fl / (ms / 1e3) / 1e12,
            "frac_fp32_peak": fl / (ms / 1e3) / PEAK["fp32"], "kernel_ms": {k: round(v, 4) for k, v in parts.items()},
            "loss": float(gb.loss.cpu()[0])}


def library_gemm_row(torch) -> dict:
    """The library's bf16 GEMM (torch.matmul, hipBLASLt) at the three products
    of one xlarge rollout step (B 16384 rows; gates K = Z + H = 1152 by
    N = 4H = 4096, mixture head K = H = 1024 by N = 3ZK = 3072, controller
    K = 1152 by N = A + 2 = 258), weights stored [N, K] as the packed layout
    holds them. A comparison for the fused kernels, which also run their
    epilogues: the GEMM alone, median over 10 batches of 20 calls."""
    res = {}
    total = 0.0
    for name, (M, K, N) in {"gates": (16384, 1152, 4096), "mixture_head": (16384, 1024, 3072),
                            "controller": (16384, 1152, 258)}.items():
        g = torch.Generator(device="cuda").manual_seed(0)
        a = torch.randn(M, K, dtype=torch.bfloat16, device="cuda", generator=g)
        w = torch.randn(N, K, dtype=torch.bfloat16, device="cuda", generator=g)
        wt = w.t()
        for _ in range(5):
            c = a @ wt
        torch.cuda.synchronize()
        times = []
        for _ in range(10):
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            for _ in range(20):
                c = a @ wt
            e.record()
            e.synchronize()
            times.append(s.elapsed_time(e) * 1e3 / 20)
        us = float(np.median(times))
        total += us
        res[name] = {"M": M, "K": K, "N": N, "us": us,
                     "frac_bf16_peak": 2.0 * M * N * K / (us * 1e-6) / PEAK["bf16"]}
        del a, w, wt, c
    res["step_gemms_us"] = total
    torch.cuda.empty_cache()
    return res


def adam_row(wmlib, torch) -> dict:
    """One optimiser step over the world model's parameters at the xlarge
    sizes (W_g 4H x (Z+A+H), W_m 3ZK x H and the biases and heads: 8.9 M fp32
    values) against the HBM roof: 16 bytes read and 12 written per value."""
    Z, H, A, K = 128, 1024, 256, 8
    n = 4 * H * (Z + A + H) + 4 * H + 3 * Z * K * H + 3 * Z * K + 2 * H + 2
    p = torch.randn(n, device="cuda")
    g = torch.randn(n, device="cuda")
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    wmlib.adam_step(p, g, m, v, 1, 1e-4)
    torch.cuda.synchronize()
    reps = 20
    wmlib.profile_reset()
    wmlib.profile_enable("adam")
    for i in range(reps):
        wmlib.adam_step(p, g, m, v, 2 + i, 1e-4)
    torch.cuda.synchronize()
    k_ms, k_n = wmlib.profile_read("adam")
    wmlib.profile_enable(None)
    wmlib.profile_reset()
    kms = k_ms / max(k_n, 1)
    nb = 28 * n
    return {"params": n, "kernel_us": kms * 1e3, "bytes": nb, "GBps": nb / (kms / 1e3) / 1e9,
            "kernel_frac_hbm_peak": nb / (kms / 1e3) / HBM_PEAK}


def two_level_row(wmlib, wl, torch, cuda, N: int = 288) -> dict:
    """A dream rollout with the two-level controller at the paper's largest
    action space (SqueezeNet1.1's 288 substitutions + NO-OP, 200 locations:
    A = 57600 world-model actions) at the large rollout's sizes (B = 4096,
    Z = 64, H = 1024, K = 8, bf16), T = 20, against the bf16 MFMA peak; the
    controller has N + 1 + L logit rows."""
    B, T, Z, H, K, L = 4096, 20, 64, 1024, 8, 200
    A = N * L
    rng = np.random.default_rng(6)
    w = wl.make_weights(rng, Z, H, A, K, T)
    a = np.sqrt(6.0 / (Z + H + N + 1 + L))
    w["W_c"] = rng.uniform(-a, a, size=(N + 1 + L, Z + H)).astype(np.float32)
    w["b_c"] = np.zeros(N + 1 + L, np.float32)
    m = wmlib.pack(w, Z, H, A, K, "bf16", N=N, L=L)
    z0 = cuda(rng.standard_normal((B, Z)).astype(np.float32))
    xm = (rng.random((B, N + 1)) < 0.5).astype(np.uint8)
    xm[:, 0] = 1
    xm[:, N] = 0
    lm = (rng.random((B, N, L)) < 0.3).astype(np.uint8)
    lm[:, :, 0] = 1
    mask = wmlib.two_level_mask(m, cuda(xm), cuda(lm))  # the library's layout, built once
    bufs = wmlib.RolloutBuffers(m, B, T)
    run = lambda i: wmlib.rollout(m, z0, mask, T=T, seed=7 + i, done=True, bufs=bufs)  # noqa: E731
    ms, reps = _median_ms(torch, run)
    fl = 2.0 * (4 * H * (Z + H) + 3 * Z * K * H + (N + 1 + L) * (Z + H) + 2 * H)
    return {"N": N, "L": L, "A": A, "ms": ms, "reps": reps, "per_s": B * T / (ms / 1e3), "unit": "transitions/s",
            "tflops": B * T * fl / (ms / 1e3) / 1e12, "frac_mfma_peak": B * T * fl / (ms / 1e3) / PEAK["bf16"]}


def returns_bytes(T: int, B: int, gae: bool) -> int:
    """Algorithmic HBM bytes of one wm_returns call: rewards (4 B) and dones
    (1 B) read and returns (4 B) written per step, plus with GAE the values
    [T+1, B] read and the advantages written."""
    return T * B * (4 + 1 + 4) + ((T + 1) * B * 4 + T * B * 4 if gae else 0)


def returns_row(wmlib, torch, cuda) -> dict:
    """GAE scan over the xlarge rollout's shape (T = 64, B = 16384), against
    the HBM roof (the kernel reads and writes each element once)."""
    T, B = 64, 16384
    rng = np.random.default_rng(5)
    r = cuda(rng.normal(size=(T, B)).astype(np.float32))
    d = cuda((rng.random((T, B)) < 0.05).astype(np.uint8))
    v = cuda(rng.normal(size=(T + 1, B)).astype(np.float32))
    out = torch.empty((T, B), dtype=torch.float32, device=r.device)
    adv = torch.empty_like(out)
    wmlib.returns(r, d, 0.99, values=v, lam=0.95, out=out, adv=adv)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 50
    a.record()
    for _ in range(reps):
        wmlib.returns(r, d, 0.99, values=v, lam=0.95, out=out, adv=adv)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    # the kernel alone: dispatch-stamped events on every launch
    wmlib.profile_reset()
    wmlib.profile_enable("returns")
    for _ in range(reps):
        wmlib.returns(r, d, 0.99, values=v, lam=0.95, out=out, adv=adv)
    torch.cuda.synchronize()
    k_ms, k_n = wmlib.profile_read("returns")
    wmlib.profile_enable(None)
    wmlib.profile_reset()
    kms = k_ms / max(k_n, 1)
    nb = returns_bytes(T, B, True)
    return {"ms": ms, "per_s": T * B / (ms / 1e3), "unit": "steps/s", "bytes": nb,
            "GBps": nb / (ms / 1e3) / 1e9, "frac_hbm_peak": nb / (ms / 1e3) / HBM_PEAK,
            "kernel_us": kms * 1e3, "kernel_frac_hbm_peak": nb / (kms / 1e3) / HBM_PEAK}


def cpu_baseline(w, roll_in, budget_s: float) -> dict:
    """The oracle as it stands (float64 numpy with the bf16 rounding points),
    timed on this host's cores on a subset of the same batch: the first
    CPU_ROWS trajectories, whole rollouts of T steps, repeated while the
    budget lasts.  A trajectory's result does not depend on the others, so
    the per-transition rate of the subset is the oracle's rate on the
    workload."""
    from oracle import wm as owm

    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        threads = int(blas[0]["num_threads"]) if blas else 1
    except Exception:  # noqa: BLE001
        threads = 1
    rows = min(CPU_ROWS, w.B)
    z0, mask = roll_in["z0"][:rows], roll_in["mask"][:rows]
    reps, t0 = 0, time.perf_counter()
    while True:
        owm.rollout(roll_in["weights"], w.dims, z0, mask, T=w.T, seed=w.seed + reps, tau=w.tau,
                    done_flag=w.done, dtype=w.dtype)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 20:
            break
    return {"value": rows * w.T * reps / el, "unit": "transitions/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{reps} whole rollout(s) of the first {rows} of the {w.B} trajectories (T={w.T}, "
                      f"{w.name}) in {el:.1f} s, float64 numpy with bf16 rounding points, "
                      f"{threads} BLAS threads, {len(os.sched_getaffinity(0))} cores visible"}


if __name__ == "__main__":
    sys.exit(main())
