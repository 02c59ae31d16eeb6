"""Summaries of rocprofv3 output for the library's kernels (host-side post-processing only).

Three summaries, each written as short text (markdown), the issue picture and the traffic
also as a JSON record:

* ``stats``: per-kernel call count and average / min / max duration from the
  ``kernel_stats.csv`` that ``rocprofv3 --kernel-trace --stats -f csv`` writes.
* ``issue``: per-kernel issue picture from one SQ counter run (``--pmc SQ_WAVES SQ_INSTS_VALU
  SQ_INSTS_MFMA SQ_INSTS_VALU_TRANS_F32 SQ_INSTS_LDS SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE``):
  the fraction of SIMD cycles in which the matrix cores are busy, and the fraction the vector
  ALU needs for the kernel's instructions: a wave64 fp32 instruction occupies a SIMD for 2
  cycles (128 lanes per clock per compute unit, the 157.3 TFLOP/s FMA rate), a
  transcendental one for 8 (a quarter of that rate). GRBM_GUI_ACTIVE is summed over the 8
  XCDs, so the kernel's cycles are its value / 8; the SIMD count is 1024.
  With ``--workload`` it also writes a JSON record of the vector-ALU and matrix-core time
  per step (each kernel's busy fraction times its duration and launches per step), which
  ``bench.py`` divides by its measured step time.
* ``traffic``: HBM bytes per launch of each kernel from two counter runs
  (``--pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``, ``-f csv``). Each counter is calibrated by
  what it reads for a plain device-to-device copy of known size that the profiled program
  issues first (``bench.py --copy-calibration-mib M``): the copy reads and writes exactly M MiB,
  so the factor is M MiB over the counter's reading for that dispatch.

The JSON record carries a hash of the kernel sources; ``bench.py`` reports the traffic only
while the hash matches the sources it runs.

Usage::

    python -m paper_2609_32525_amd.profiling stats DIR/kernel_stats.csv --command "..." --out F.md
    python -m paper_2609_32525_amd.profiling issue DIR --command "..." --out F.md
    python -m paper_2609_32525_amd.profiling traffic FETCH_DIR WRITE_DIR --copy-mib 256 \
        --workload surface --command "..." --out profiles/pmc_<kernel>_<workload>
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re
import subprocess
from typing import Dict, List, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("fs_stream.h", "fs_pass_slice.hip", "fs_pass_deslice.hip", "fs_pass_bwd_a.hip",
                  "fs_pass_bwd_b.hip", "fs_pass_point.hip", "fs_pass_linearno.hip", "fs_pass_bwd_b2.hip", "fs_kernels.hip", "fs_tokens.hip", "fs_tokmix.hip",
                  "fs_api.cpp", "fs_internal.h")
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def kernel_source_hash() -> str:
    """First 16 hex digits of the SHA-256 of the kernel and launcher sources, with line
    comments and blank lines removed (editing a comment does not change a kernel)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(_HERE, "csrc", f)) as fh:
            for line in fh:
                code = re.sub(r"//.*$", "", line).rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


def short_name(name: str) -> str:
    """Demangled kernel name without namespaces, argument list and return type."""
    if name.startswith("_Z"):
        try:
            name = subprocess.run(["c++filt", name], capture_output=True, text=True,
                                  check=True).stdout.strip()
        except (OSError, subprocess.CalledProcessError):
            pass
    name = re.sub(r"fs::\(anonymous namespace\)::|fs::", "", name)
    name = re.sub(r"^void ", "", name)
    depth, cut = 0, len(name)
    for i, c in enumerate(name):      # drop the argument list: first '(' outside <...>
        if c == "<":
            depth += 1
        elif c == ">":
            depth -= 1
        elif c == "(" and depth == 0:
            cut = i
            break
    return name[:cut].strip()


def _find(path: str, pattern: str) -> str:
    if os.path.isfile(path):
        return path
    hits = glob.glob(os.path.join(path, "**", pattern), recursive=True)
    if not hits:
        raise FileNotFoundError(f"no {pattern} under {path}")
    return max(hits, key=os.path.getmtime)  # the latest run's file


def kernel_stats(path: str) -> List[Tuple[str, int, float, float, float, float]]:
    """(kernel, calls, total_us, avg_us, min_us, max_us) sorted by total time."""
    rows = []
    with open(_find(path, "*kernel_stats.csv")) as fh:
        for r in csv.DictReader(fh):
            ns = 1e-3
            rows.append((short_name(r["Name"]), int(r["Calls"]), float(r["TotalDurationNs"]) * ns,
                         float(r["AverageNs"]) * ns, float(r["MinNs"]) * ns,
                         float(r["MaxNs"]) * ns))
    rows.sort(key=lambda t: -t[2])
    return rows


def counter_values(path: str, counter: str) -> Dict[str, List[float]]:
    """Per-dispatch values (KiB for FETCH_SIZE / WRITE_SIZE) of one counter, by kernel."""
    per_dispatch: Dict[Tuple[str, str], float] = collections.defaultdict(float)
    with open(_find(path, "*counter_collection.csv")) as fh:
        for r in csv.DictReader(fh):
            if r["Counter_Name"] != counter:
                continue
            per_dispatch[(r["Dispatch_Id"], r["Kernel_Name"])] += float(r["Counter_Value"])
    out: Dict[str, List[float]] = collections.defaultdict(list)
    for (_, k), v in sorted(per_dispatch.items(), key=lambda kv: int(kv[0][0])):
        out[k].append(v)
    return out


ISSUE_COUNTERS = ("SQ_WAVES", "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_VALU_TRANS_F32",
                  "SQ_INSTS_LDS", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
SIMDS, XCDS = 1024, 8
VALU_CYCLES, TRANS_CYCLES = 2.0, 8.0  # SIMD cycles per wave64 instruction


def issue_summary(path: str) -> Dict[str, Dict[str, float]]:
    """Per kernel, averaged over its dispatches: cycles, waves, instruction counts, the
    MFMA-busy and VALU-issue fractions of the SIMD cycles, and the implied clock."""
    per: Dict[Tuple[str, str], Dict[str, float]] = collections.defaultdict(
        lambda: collections.defaultdict(float))
    dur: Dict[Tuple[str, str], float] = {}
    with open(_find(path, "*counter_collection.csv")) as fh:
        for r in csv.DictReader(fh):
            key = (r["Dispatch_Id"], short_name(r["Kernel_Name"]))
            per[key][r["Counter_Name"]] += float(r["Counter_Value"])
            dur[key] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    agg: Dict[str, Dict[str, float]] = collections.defaultdict(lambda: collections.defaultdict(float))
    for (d, k), cs in per.items():
        if k.startswith(("__amd", "at::")):
            continue
        a = agg[k]
        a["n"] += 1
        a["ns"] += dur[(d, k)]
        for c, v in cs.items():
            a[c] += v
    out = {}
    for k, a in agg.items():
        n = a["n"]
        cyc = a["GRBM_GUI_ACTIVE"] / n / XCDS
        simd_cyc = max(cyc * SIMDS, 1.0)
        out[k] = {"dispatches": n, "us": a["ns"] / n * 1e-3, "cycles": cyc,
                  "clock_ghz": cyc / max(a["ns"] / n, 1.0),
                  "waves": a["SQ_WAVES"] / n, "valu_insts": a["SQ_INSTS_VALU"] / n,
                  "mfma_insts": a["SQ_INSTS_MFMA"] / n, "lds_insts": a["SQ_INSTS_LDS"] / n,
                  "trans_insts": a["SQ_INSTS_VALU_TRANS_F32"] / n,
                  "mfma_busy": a["SQ_VALU_MFMA_BUSY_CYCLES"] / n / simd_cyc,
                  # SQ_INSTS_VALU counts MFMAs too; they run on the matrix cores
                  "valu_busy": (VALU_CYCLES * (a["SQ_INSTS_VALU"] - a["SQ_INSTS_MFMA"]
                                               - a["SQ_INSTS_VALU_TRANS_F32"])
                                + TRANS_CYCLES * a["SQ_INSTS_VALU_TRANS_F32"]) / n / simd_cyc}
    return out


def issue_record(res: Dict[str, Dict[str, float]], workload: str, command: str) -> dict:
    """Per-step vector-ALU and matrix-core time from an issue summary: each kernel's SIMD
    cycles of VALU issue (valu_busy x its cycles) and of MFMA busy, over the 1024 SIMDs at
    its measured clock, times its launches per step. Launches per step are counted against
    the deslice, which every step of the path launches exactly once."""
    steps = max((r["dispatches"] for k, r in res.items() if k.startswith("k_deslice")),
                default=0)
    if steps == 0:
        raise RuntimeError("no deslice dispatches to count steps by")
    kernels = {}
    t_valu = t_mfma = 0.0
    for k, r in res.items():
        per_step = r["dispatches"] / steps
        tv = r["valu_busy"] * r["us"]
        tm = r["mfma_busy"] * r["us"]
        kernels[k] = {"launches_per_step": per_step, "us": r["us"], "valu_busy": r["valu_busy"],
                      "mfma_busy": r["mfma_busy"], "t_valu_us": tv, "t_mfma_us": tm}
        t_valu += tv * per_step
        t_mfma += tm * per_step
    return {"workload": workload, "kernel_source_sha256": kernel_source_hash(),
            "t_valu_us_per_step": t_valu, "t_mfma_us_per_step": t_mfma,
            "valu_cycles_per_inst": VALU_CYCLES, "trans_cycles_per_inst": TRANS_CYCLES,
            "kernels": kernels, "command": command}


def calibrated_traffic(fetch_dir: str, write_dir: str, copy_mib: float):
    """Per-kernel average (fetch, write) bytes per launch, each counter scaled by its reading
    for the copy of ``copy_mib`` MiB (only copy dispatches of at least half that size count)."""
    f = counter_values(fetch_dir, "FETCH_SIZE")
    w = counter_values(write_dir, "WRITE_SIZE")
    kib = copy_mib * 1024.0

    def scale(vals, what):
        big = [v for v in vals if v > 0.5 * kib]
        if not big:
            raise RuntimeError(f"no calibration copy of {copy_mib} MiB in the {what} run")
        return kib / (sum(big) / len(big))

    cf = scale([v for k, vs in f.items() if short_name(k) == COPY_KERNEL for v in vs], "fetch")
    cw = scale([v for k, vs in w.items() if short_name(k) == COPY_KERNEL for v in vs], "write")
    res = {}
    for k in f:
        if short_name(k).startswith(("__amd", "at::")) or k not in w:
            continue
        fb = sum(f[k]) / len(f[k]) * cf * 1024.0
        wb = sum(w[k]) / len(w[k]) * cw * 1024.0
        res[short_name(k)] = {"fetch_bytes": fb, "write_bytes": wb, "dispatches": len(f[k])}
    return cf, cw, res


def _main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("path")
    s.add_argument("--command", required=True, help="the rocprofv3 command that made it")
    s.add_argument("--title", default="Kernel durations")
    s.add_argument("--out", required=True)
    q = sub.add_parser("issue")
    q.add_argument("path")
    q.add_argument("--command", required=True)
    q.add_argument("--title", default="Issue picture")
    q.add_argument("--out", required=True)
    q.add_argument("--workload", default=None,
                   help="also write a JSON record (OUT with .json) that bench.py reads")
    t = sub.add_parser("traffic")
    t.add_argument("fetch")
    t.add_argument("write")
    t.add_argument("--copy-mib", type=float, required=True)
    t.add_argument("--workload", required=True)
    t.add_argument("--kernel", action="append",
                   help="kernel(s) whose summed traffic the JSON record holds (default k_bwd_b; "
                        "a pass made of two kernels, such as the slot-blocked pass B, names both)")
    t.add_argument("--command", action="append", required=True)
    t.add_argument("--out", required=True, help="output path without extension")
    a = ap.parse_args()

    if a.cmd == "stats":
        rows = kernel_stats(a.path)
        tot = sum(r[2] for r in rows) or 1.0
        lines = [f"# {a.title}", "", "Command:", "", "```", a.command, "```", "",
                 f"Kernel sources sha256[:16] = `{kernel_source_hash()}`", "",
                 "| kernel | calls | avg us | min us | max us | % time |",
                 "|---|---:|---:|---:|---:|---:|"]
        for n, c, tt, av, mn, mx in rows:
            if n.startswith("at::"):
                continue
            lines.append(f"| `{n}` | {c} | {av:.2f} | {mn:.2f} | {mx:.2f} | {100 * tt / tot:.1f} |")
        with open(a.out, "w") as fh:
            fh.write("\n".join(lines) + "\n")
        print("\n".join(lines))
        return

    if a.cmd == "issue":
        res = issue_summary(a.path)
        lines = [f"# {a.title}", "", "Command:", "", "```", a.command, "```", "",
                 f"Kernel sources sha256[:16] = `{kernel_source_hash()}`", "",
                 "MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES over the SIMD cycles (1024 SIMDs x the "
                 "kernel's cycles, GRBM_GUI_ACTIVE / 8 XCDs). VALU busy: the vector instructions "
                 "(SQ_INSTS_VALU less the MFMAs) at 2 SIMD cycles each, transcendentals "
                 "(SQ_INSTS_VALU_TRANS_F32) at 8, over the same SIMD cycles. Idle: the SIMD "
                 "time neither accounts for (waiting on memory, LDS or barriers, or on dependent "
                 "results), taking MFMA and VALU work as overlapping perfectly.", "",
                 "| kernel | us | waves | VALU / wave | exp / wave | MFMA / wave | "
                 "LDS / wave | MFMA busy | VALU busy | idle |",
                 "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
        for k, r in sorted(res.items(), key=lambda kv: -kv[1]["us"]):
            w = max(r["waves"], 1.0)
            idle = max(0.0, 1.0 - max(r["mfma_busy"], r["valu_busy"]))
            lines.append(f"| `{k}` | {r['us']:.1f} | {r['waves']:.0f} | "
                         f"{(r['valu_insts'] - r['mfma_insts']) / w:.0f} | "
                         f"{r['trans_insts'] / w:.0f} | {r['mfma_insts'] / w:.0f} | "
                         f"{r['lds_insts'] / w:.0f} | {100 * r['mfma_busy']:.1f}% | "
                         f"{100 * r['valu_busy']:.1f}% | {100 * idle:.0f}% |")
        with open(a.out, "w") as fh:
            fh.write("\n".join(lines) + "\n")
        print("\n".join(lines))
        if a.workload:
            rec = issue_record(res, a.workload, a.command)
            with open(os.path.splitext(a.out)[0] + ".json", "w") as fh:
                json.dump(rec, fh, indent=1)
        return

    cf, cw, res = calibrated_traffic(a.fetch, a.write, a.copy_mib)
    lines = [f"# HBM traffic per launch, workload {a.workload}", "",
             "Commands (one counter per run):", "", "```"] + a.command + ["```", "",
             f"Calibration: a {a.copy_mib:g} MiB device copy; FETCH_SIZE x{cf:.3f}, "
             f"WRITE_SIZE x{cw:.3f}.", "",
             f"Kernel sources sha256[:16] = `{kernel_source_hash()}`", "",
             "| kernel | dispatches | fetch MiB | write MiB |", "|---|---:|---:|---:|"]
    for n, r in res.items():
        lines.append(f"| `{n}` | {r['dispatches']} | {r['fetch_bytes'] / 2**20:.2f} | "
                     f"{r['write_bytes'] / 2**20:.2f} |")
    with open(a.out + ".md", "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    kernels = a.kernel or ["k_bwd_b"]
    mine = [n for n in res if any(n.startswith(k + "<") or n == k for k in kernels)]
    if mine:
        fb = sum(res[n]["fetch_bytes"] for n in mine)
        wb = sum(res[n]["write_bytes"] for n in mine)
        rec = {"workload": a.workload, "kernel": " + ".join(mine),
               "kernel_source_sha256": kernel_source_hash(),
               "fetch_scale": cf, "write_scale": cw, "copy_mib": a.copy_mib,
               "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
               "traffic_bytes_per_launch": fb + wb, "commands": a.command}
        with open(a.out + ".json", "w") as fh:
            json.dump(rec, fh, indent=1)


if __name__ == "__main__":
    _main()
