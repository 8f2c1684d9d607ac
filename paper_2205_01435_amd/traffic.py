"""rocprofv3 counter runs and their summaries.

HBM traffic per launch of one kernel class comes from two rocprofv3 passes
over the same program (one pass per counter, as the hardware collects
FETCH_SIZE and WRITE_SIZE on the same TCC blocks):

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/fetch -o run -- \
        python3 -m paper_2205_01435_amd.traffic run --workload xlarge_rollout
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/write -o run -- \
        python3 -m paper_2205_01435_amd.traffic run --workload xlarge_rollout
    python3 -m paper_2205_01435_amd.traffic summarize OUT/fetch/run_counter_collection.csv \
        OUT/write/run_counter_collection.csv --kernel k_gates --workload xlarge_rollout \
        --out profiles/<file>.md

``run`` first copies 256 MiB device to device three times (a copy kernel that
reads and writes exactly that many bytes: the calibration of each counter),
then runs calls of one workload (default: two of the xlarge dream rollout).
``summarize`` scales the kernel's per-dispatch average by bytes / counter of
the copy and writes a short summary, stamped with the names and hash of the
sources the kernel is compiled from, so that a reader (bench.py) can tell
whether the figures still describe the current kernel.

``counters`` summarises any other counters of a ``--pmc`` pass (per-dispatch
averages of the kernels a regex selects), and ``stats`` a
``--kernel-trace --stats`` run's kernel_stats.csv.
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
XCDS, SIMDS = 8, 1024  # MI355X: 8 XCDs, 256 CUs x 4 SIMDs


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


def run(workload: str = "xlarge_rollout", calls: int = 2) -> None:
    """The calibration copies, then ``calls`` calls of one workload (a dream
    rollout or an NLL pass) on its seeded inputs."""
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

    w = wl.WORKLOADS[workload]
    cuda = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    if w.kind == "rollout":
        inp = wl.make_rollout_inputs(w)
        model = wmlib.pack(inp["weights"], w.Z, w.H, w.A, w.K, w.dtype)
        z0, mask = cuda(inp["z0"]), cuda(inp["mask"])
        rb = wmlib.RolloutBuffers(model, w.B, w.T, trace=False)
        for i in range(calls):
            wmlib.rollout(model, z0, mask, T=w.T, seed=w.seed + i, tau=w.tau, done=w.done, bufs=rb)
            torch.cuda.synchronize()
            print(f"{workload}: call {i + 1} of {calls} done", flush=True)
    else:
        d = wl.make_nll_inputs(w)
        model = wmlib.pack(d["weights"], w.Z, w.H, w.A, w.K, w.dtype)
        args = [cuda(d[k]) for k in ("z", "actions", "rewards", "dones")]
        nb = wmlib.NllBuffers(model, w.B, w.T)
        for i in range(calls):
            wmlib.nll(model, *args, bufs=nb)
            torch.cuda.synchronize()
            print(f"{workload}: call {i + 1} of {calls} done", flush=True)
    print("counter run done", flush=True)


def _per_dispatch(path: str, counter: str) -> list[tuple[str, int, float]]:
    """(kernel name, grid size, counter value) per dispatch."""
    rows = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            rows.append((r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])))
    return rows


def summarize(fetch_csv: str, write_csv: str, kernel: str, out: str, command: str,
              workload: str = "") -> dict:
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
        f"# HBM traffic per launch: {kernel} ({workload or 'workload not named'})",
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


def counters(csvs: list[str], kernel: str, out: str, title: str, command: str, note: str = "") -> dict:
    """Per-dispatch averages of every counter in the given counter-collection
    CSVs over the dispatches whose kernel name matches ``kernel``."""
    acc: dict[tuple[str, str], list[float]] = {}
    for path in csvs:
        with open(path, newline="") as f:
            for r in csv.DictReader(f):
                if not re.search(kernel, r["Kernel_Name"]):
                    continue
                acc.setdefault((r["Kernel_Name"], r["Counter_Name"]), []).append(float(r["Counter_Value"]))
    if not acc:
        raise SystemExit(f"no dispatch of {kernel} in {csvs}")
    lines = [f"# {title}", "", f"command: `{command}`", ""]
    if note:
        lines += [note, ""]
    lines += ["| kernel | counter | dispatches | average per dispatch |", "|---|---|---|---|"]
    res = {}
    for (k, c), v in sorted(acc.items()):
        avg = sum(v) / len(v)
        res.setdefault(k, {})[c] = avg
        lines.append(f"| `{_short(k)}` | {c} | {len(v)} | {avg:.6g} |")
    derived = []
    for k, cs in res.items():
        # GRBM_GUI_ACTIVE is summed over the 8 XCDs; the SQ counters over all 1024 SIMDs
        if "SQ_VALU_MFMA_BUSY_CYCLES" in cs and cs.get("GRBM_GUI_ACTIVE"):
            cyc = cs["GRBM_GUI_ACTIVE"] / XCDS
            derived.append((k, "MFMA busy, % of SIMD cycles", 100.0 * cs["SQ_VALU_MFMA_BUSY_CYCLES"] / SIMDS / cyc))
            if "SQ_INSTS_VALU" in cs:
                other = cs["SQ_INSTS_VALU"] - cs.get("SQ_INSTS_MFMA", 0.0)
                derived.append((k, "non-MFMA VALU instructions per SIMD", other / SIMDS))
                derived.append((k, "their issue cycles (4 per wave64 instruction), % of SIMD cycles",
                                100.0 * 4 * other / SIMDS / cyc))
            derived.append((k, "kernel cycles per XCD (GRBM_GUI_ACTIVE / 8)", cyc))
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in cs:
            derived.append((k, "bf16 MFMA flops (MOPS x 512)", 512.0 * cs["SQ_INSTS_VALU_MFMA_MOPS_BF16"]))
        if "TCC_HIT_sum" in cs and "TCC_MISS_sum" in cs:
            tot = cs["TCC_HIT_sum"] + cs["TCC_MISS_sum"]
            derived.append((k, "L2 hit rate, %", 100.0 * cs["TCC_HIT_sum"] / tot if tot else 0.0))
    if derived:
        lines += ["", "| kernel | derived | value |", "|---|---|---|"]
        for k, name, v in derived:
            res[k][name] = v
            lines.append(f"| `{_short(k)}` | {name} | {v:.6g} |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    return res


def _short(name: str, n: int = 90) -> str:
    return name if len(name) <= n else name[:n - 1] + "\u2026"


def stats(csv_path: str, out: str, title: str, command: str, note: str = "", top: int = 14) -> list:
    """A kernel_stats.csv of `rocprofv3 --kernel-trace --stats` as a table."""
    rows = []
    with open(csv_path, newline="") as f:
        for r in csv.DictReader(f):
            rows.append((r["Name"], int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                         float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    rows.sort(key=lambda x: -x[5])
    lines = [f"# {title}", "", f"command: `{command}`", ""]
    if note:
        lines += [note, ""]
    lines += ["| kernel | calls | avg us | min us | max us | share % |", "|---|---|---|---|---|---|"]
    for name, calls, avg, mn, mx, pct in rows[:top]:
        lines.append(f"| `{_short(name)}` | {calls} | {avg:.2f} | {mn:.2f} | {mx:.2f} | {pct:.1f} |")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    return rows


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    r = sub.add_parser("run")
    r.add_argument("--workload", default="xlarge_rollout")
    r.add_argument("--calls", type=int, default=2)
    s = sub.add_parser("summarize")
    s.add_argument("fetch_csv")
    s.add_argument("write_csv")
    s.add_argument("--kernel", required=True, help="regex on the kernel name")
    s.add_argument("--workload", default="")
    s.add_argument("--out", required=True)
    s.add_argument("--command", default="", help="command line to record in the summary")
    c = sub.add_parser("counters")
    c.add_argument("csvs", nargs="+")
    c.add_argument("--kernel", required=True, help="regex on the kernel name")
    c.add_argument("--out", required=True)
    c.add_argument("--title", required=True)
    c.add_argument("--command", default="")
    c.add_argument("--note", default="")
    t = sub.add_parser("stats")
    t.add_argument("csv")
    t.add_argument("--out", required=True)
    t.add_argument("--title", required=True)
    t.add_argument("--command", default="")
    t.add_argument("--note", default="")
    a = ap.parse_args()
    if a.cmd == "run":
        run(a.workload, a.calls)
    elif a.cmd == "summarize":
        print(summarize(a.fetch_csv, a.write_csv, a.kernel, a.out, a.command, a.workload))
    elif a.cmd == "counters":
        print(counters(a.csvs, a.kernel, a.out, a.title, a.command, a.note))
    else:
        stats(a.csv, a.out, a.title, a.command, a.note)
    return 0


if __name__ == "__main__":
    sys.exit(main())
