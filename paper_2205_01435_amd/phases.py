"""Per-phase timing of the persistent kernels (wm_profile_phases).

    python3 -m paper_2205_01435_amd.phases --workload tiny_rollout --out profiles/<file>.md

runs one workload served by the persistent kernels (the tiny and medium
dream rollouts, the NLL pass) with phase stamps on, a few warm-up calls and
then ``--calls`` stamped calls, and writes the median of each slot over the
calls (microseconds per step) as a short markdown summary.  The stamps are
the device's constant-rate clock, taken by one lane of each work-group at
the start, at each arrival at and release from an XCD barrier, and at the
end of the launch.
"""

from __future__ import annotations

import argparse
import statistics
import sys

import numpy as np
import torch

from . import _lib as wmlib
from . import workloads as wl

DESCR = {
    "step": "wall time per step (first release of the set-up barrier to that of the last step's)",
    "gates": "gates(t): staging, gate MFMAs, controller decisions, LSTM cell (max over an XCD's "
             "work-groups); NLL: the step",
    "gates_barrier": "barrier after gates(t): last arrival to first release (the mixture noise is drawn in it)",
    "mdn": "mdn(t): mixture head, component pick, Box-Muller, z commit, next controller h part (max)",
    "mdn_barrier": "barrier after mdn(t) (the controller's Gumbel noise is drawn in it)",
    "gates_mean": "gates(t), mean",
    "mdn_mean": "mdn(t), mean",
    "setup": "set-up: register weights, LDS tables, step-0 controller h part (max, once per call)",
    "tail": "tail: the last transition's reward and done, final cell state (max, once per call)",
}


def measure(name: str, calls: int = 20, warmup: int = 3) -> dict:
    w = wl.WORKLOADS[name]
    if w.kind == "rollout":
        inp = wl.make_rollout_inputs(w)
        m = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
        z0 = torch.from_numpy(inp["z0"]).cuda()
        mask = torch.from_numpy(inp["mask"]).cuda()
        bufs = wmlib.RolloutBuffers(m, w.B, w.T)

        def call(i):
            wmlib.rollout(m, z0, mask, T=w.T, seed=w.seed + i, done=w.done, bufs=bufs)
    else:
        d = wl.make_nll_inputs(w)
        m = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, w.dtype)
        args = [torch.from_numpy(np.ascontiguousarray(d[k])).cuda() for k in ("z", "actions", "rewards", "dones")]
        bufs = wmlib.NllBuffers(m, w.B, w.T)

        def call(i):
            wmlib.nll(m, *args, bufs=bufs)
    for i in range(warmup):
        call(i)
    torch.cuda.synchronize()
    rows = []
    wmlib.profile_phases(True)
    try:
        for i in range(calls):
            call(i)
            r = wmlib.profile_phases_read()
            if r["T"] == 0:
                raise RuntimeError(f"{name}: no persistent launch was stamped (not served by the persistent kernels)")
            rows.append(r)
    finally:
        wmlib.profile_phases(False)
    return {k: statistics.median(r[k] for r in rows) for k in wmlib.PHASE_SLOTS}


def summary(name: str, res: dict, calls: int) -> str:
    w = wl.WORKLOADS[name]
    cmd = f"python3 -m paper_2205_01435_amd.phases --workload {name} --calls {calls} --out <this file>"
    lines = [f"# Persistent-kernel phases: {name} (B {w.B}, T {w.T}, Z {w.Z}, H {w.H}, A {w.A}, K {w.K}, {w.dtype})",
             "", f"Command: `{cmd}`", "",
             f"Median over {calls} stamped calls of each slot, microseconds per step (set-up and tail: per call).",
             "", "| slot | us | what |", "|---|---:|---|"]
    for k in wmlib.PHASE_SLOTS[1:]:
        if k in ("ctrl", "ctrl_barrier", "ctrl_mean"):
            continue  # the controller decisions run inside gates(t)
        if w.kind == "nll" and k in ("mdn", "mdn_barrier", "mdn_mean", "tail"):
            continue
        lines.append(f"| {k} | {res[k]:.3f} | {DESCR[k]} |")
    parts = ("gates", "gates_barrier", "mdn", "mdn_barrier")
    acc = sum(res[k] for k in parts)
    lines += ["", f"Sum of the max-work and barrier slots: {acc:.3f} us of the {res['step']:.3f} us step "
              "(the rest is skew: work-groups leave a barrier at different times).", ""]
    return "\n".join(lines)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--workload", default="tiny_rollout")
    ap.add_argument("--calls", type=int, default=20)
    ap.add_argument("--out", default=None)
    a = ap.parse_args(argv)
    assert torch.cuda.is_available(), "phase timing needs the GPU"
    wmlib.load()
    res = measure(a.workload, a.calls)
    text = summary(a.workload, res, a.calls)
    print(text, flush=True)
    if a.out:
        with open(a.out, "w") as f:
            f.write(text)
    return 0


if __name__ == "__main__":
    sys.exit(main())
