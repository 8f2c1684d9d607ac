"""HBM traffic per launch of one kernel class, from rocprofv3 counters.

The counters come from two rocprofv3 passes over the same program (one pass
per counter, as the hardware collects FETCH_SIZE and WRITE_SIZE on the same
TCC blocks):

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/fetch -o run -- \
        python3 -m paper_2205_01435_amd.traffic run
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/write -o run -- \
        python3 -m paper_2205_01435_amd.traffic run
    python3 -m paper_2205_01435_amd.traffic summarize OUT/fetch/run_counter_collection.csv \
        OUT/write/run_counter_collection.csv --kernel k_gates --out profiles/<file>.md

``run`` first copies 256 MiB device to device three times (a copy kernel that
reads and writes exactly that many bytes: the calibration of each counter),
then runs two bench steps (medium dream rollout + NLL).  ``summarize`` scales
the kernel's per-dispatch average by bytes / counter of the copy and writes a
short summary, stamped with the names and hash of the sources the kernel is
compiled from, so that a reader (bench.py) can tell whether the figures still
describe the current kernel.
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
HEADERS = ["wm_device.h", "wm_kernels.h", "wm_layout.h"]
CALIB_BYTES = 256 << 20


def kernel_sources(kernel: str) -> list[str]:
    """The sources a kernel is compiled from: the persistent kernels live in
    wm_persist.hip, every other kernel in wm_kernels.hip."""
    return ["wm_persist.hip" if "persist" in kernel else "wm_kernels.hip", *HEADERS]


def kernel_source_hash(sources: list[str]) -> str:
    """sha256 over the given kernel sources."""
    h = hashlib.sha256()
    for name in sources:
        with open(os.path.join(PKG, "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def run() -> None:
    import numpy as np
    import torch

    from . import _lib as wmlib
    from . import workloads as wl

    torch.cuda.set_device(0)
    a = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device="cuda").uniform_()
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    del a, b

    w = wl.WORKLOADS["medium_rollout"]
    roll = wl.make_rollout_inputs(w)
    nll_in = wl.make_nll_inputs(w.replace(kind="nll"))
    cuda = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    model = wmlib.pack(roll["weights"], w.Z, w.H, w.A, w.K, w.dtype)
    z0, mask = cuda(roll["z0"]), cuda(roll["mask"])
    nz, na, nr, nd = (cuda(nll_in[k]) for k in ("z", "actions", "rewards", "dones"))
    rb = wmlib.RolloutBuffers(model, w.B, w.T, trace=False)
    nb = wmlib.NllBuffers(model, w.B, w.T)
    for i in range(2):
        wmlib.rollout(model, z0, mask, T=w.T, seed=w.seed + i, tau=w.tau, done=w.done, bufs=rb)
        wmlib.nll(model, nz, na, nr, nd, bufs=nb)
    torch.cuda.synchronize()
    print("traffic run done", flush=True)


def _per_dispatch(path: str, counter: str) -> list[tuple[str, int, float]]:
    """(kernel name, grid size, counter value) per dispatch."""
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            rows.append((r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])))
    return rows


def summarize(fetch_csv: str, write_csv: str, kernel: str, out: str, command: str) -> dict:
    res = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = _per_dispatch(path, counter)
        calib = [v for name, _, v in rows if "copyBuffer" in name and v * 1024 > CALIB_BYTES / 2]
        mine = [v for name, _, v in rows if re.search(kernel, name)]
        if not calib or not mine:
            raise SystemExit(f"{counter}: no calibration copy or no {kernel} dispatch in {path}")
        kib_copy = sum(calib) / len(calib)
        kib_kernel = sum(mine) / len(mine)
        factor = CALIB_BYTES / (kib_copy * 1024.0)
        res[counter] = {"kib_per_dispatch": kib_kernel, "dispatches": len(mine),
                        "copy_kib": kib_copy, "factor": factor,
                        "bytes_per_launch": kib_kernel * 1024.0 * factor}
    total = res["FETCH_SIZE"]["bytes_per_launch"] + res["WRITE_SIZE"]["bytes_per_launch"]
    lines = [
        f"# HBM traffic per launch: {kernel} (medium dream rollout + NLL, fp32)",
        "",
        "Counters from two `rocprofv3 --pmc` passes (FETCH_SIZE, then WRITE_SIZE, KiB per",
        f"dispatch), each scaled by bytes / counter of a {CALIB_BYTES >> 20} MiB device copy",
        "in the same program.",
        "",
        f"command: `{command}`",
        "",
        "| counter | KiB / dispatch | dispatches | copy KiB | factor | bytes / launch |",
        "|---|---|---|---|---|---|",
    ]
    for c, r in res.items():
        lines.append(f"| {c} | {r['kib_per_dispatch']:.1f} | {r['dispatches']} | {r['copy_kib']:.0f} | "
                     f"{r['factor']:.4f} | {r['bytes_per_launch']:.0f} |")
    srcs = kernel_sources(kernel)
    lines += ["", f"traffic_bytes_per_launch: {total:.0f}",
              f"kernel_sources: {','.join(srcs)}",
              f"kernel_source_sha256: {kernel_source_hash(srcs)}", ""]
    os.makedirs(os.path.dirname(os.path.abspath(out)), exist_ok=True)
    with open(out, "w") as f:
        f.write("\n".join(lines))
    return {"traffic_bytes_per_launch": total, **res}


def read_summary(path: str) -> float | None:
    """Bytes per launch from a summary, or None if it is missing or was taken
    on a kernel whose sources have changed since."""
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"^traffic_bytes_per_launch: (\S+)$", text, re.M)
    srcs = re.search(r"^kernel_sources: (\S+)$", text, re.M)
    h = re.search(r"^kernel_source_sha256: (\S+)$", text, re.M)
    if not m or not srcs or not h:
        return None
    names = srcs.group(1).split(",")
    if any(not os.path.exists(os.path.join(PKG, "csrc", n)) for n in names):
        return None
    if h.group(1) != kernel_source_hash(names):
        return None
    return float(m.group(1))


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    sub.add_parser("run")
    s = sub.add_parser("summarize")
    s.add_argument("fetch_csv")
    s.add_argument("write_csv")
    s.add_argument("--kernel", required=True, help="regex on the kernel name")
    s.add_argument("--out", required=True)
    s.add_argument("--command", default="", help="command line to record in the summary")
    a = ap.parse_args()
    if a.cmd == "run":
        run()
    else:
        print(summarize(a.fetch_csv, a.write_csv, a.kernel, a.out, a.command))
    return 0


if __name__ == "__main__":
    sys.exit(main())
