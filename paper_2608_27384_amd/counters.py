"""Summaries of rocprofv3 output for the measurement record (no GPU work).

Two uses:

* ``stats``: the per-kernel table of ``rocprofv3 --kernel-trace --stats
  --output-format csv`` (``*_kernel_stats.csv``), shortened to the kernels
  that matter, as text.
* ``bytes``: HBM bytes per launch of one kernel from two counter runs of
  ``bench.py --pmc-driver STAGE``, one with ``--pmc FETCH_SIZE`` and one with
  ``--pmc WRITE_SIZE`` (``*_counter_collection.csv``, KiB per dispatch).  The
  driver launches the stage 20 times and then copies 256 MiB device to
  device once; what each counter reads for that copy, against the 256 MiB it
  really moved, is the factor that turns the counter into bytes.  The summary
  records a digest of the kernel's source files so that a reader (bench.py)
  can tell when the kernel has changed since the counters were taken.

python -m paper_2608_27384_amd.counters stats CSV [--top N] [--cmd TEXT]
python -m paper_2608_27384_amd.counters bytes --fetch CSV --write CSV --stage NAME
       --workload NAME [--cmd TEXT ...]
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re
import sys
from typing import Dict, List, Optional, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
PROFILES = os.path.join(ROOT, "profiles")

COPY_BYTES = 256 << 20          # the driver's calibration copy
DRIVER_LAUNCHES = 20            # stage launches the driver makes

# stage -> (substring of the kernel's mangled name, source files that define it)
KERNELS: Dict[str, Tuple[str, Tuple[str, ...]]] = {
    "film_maps": ("EpiBiasF32", ("csrc/fv_gemm.hip", "csrc/fv_internal.h")),
    "qkv_gemm": ("EpiQkv", ("csrc/fv_gemm.hip", "csrc/fv_internal.h")),
    "attention": ("attn16d_kernel", ("csrc/fv_attn.hip", "csrc/fv_internal.h")),
    "attn_combine": ("attn_combine", ("csrc/fv_attn.hip", "csrc/fv_internal.h")),
    "gate_up_gemm": ("EpiGeglu", ("csrc/fv_gemm.hip", "csrc/fv_internal.h")),
}


def short_name(name: str) -> str:
    name = re.sub(r"fv::\(anonymous namespace\)::", "", name)
    name = re.sub(r"fv::", "", name)
    return re.sub(r"\(.*", "", name)


def source_digest(stage: str) -> str:
    h = hashlib.sha256()
    for rel in KERNELS[stage][1]:
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _rows(path: str) -> List[dict]:
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _kib(rows: List[dict], counter: str) -> List[Tuple[str, float]]:
    out = [(r["Kernel_Name"], float(r["Counter_Value"])) for r in rows
           if r.get("Counter_Name") == counter]
    if not out:
        raise ValueError(f"no {counter} rows")
    return out


def _kernel_mean(vals: List[Tuple[str, float]], sub: str) -> Tuple[float, int]:
    mine = [v for n, v in vals if sub in n]
    if len(mine) < DRIVER_LAUNCHES:
        raise ValueError(f"{len(mine)} dispatches of *{sub}* (want >= {DRIVER_LAUNCHES})")
    last = mine[-DRIVER_LAUNCHES:]
    return sum(last) / len(last), len(last)


def _copy_kib(vals: List[Tuple[str, float]]) -> float:
    cp = [v for n, v in vals if "copyBuffer" in n]
    if not cp:
        raise ValueError("no copy dispatch found")
    return max(cp)


def bytes_summary(fetch_csv: str, write_csv: str, stage: str, workload: str,
                  cmds: List[str]) -> str:
    sub = KERNELS[stage][0]
    fv, wv = _kib(_rows(fetch_csv), "FETCH_SIZE"), _kib(_rows(write_csv), "WRITE_SIZE")
    f_kib, n = _kernel_mean(fv, sub)
    w_kib, _ = _kernel_mean(wv, sub)
    cf, cw = _copy_kib(fv), _copy_kib(wv)
    f_scale = COPY_BYTES / (cf * 1024.0)
    w_scale = COPY_BYTES / (cw * 1024.0)
    fetch_b = f_kib * 1024.0 * f_scale
    write_b = w_kib * 1024.0 * w_scale
    lines = [
        f"# HBM bytes per launch: {stage} ({sub}), workload {workload}",
        "",
        "commands (repo root; rocprofv3 run from /tmp with TMPDIR=/tmp):",
        *[f"  {c}" for c in cmds],
        "",
        f"kernel_match: {sub}",
        f"stage: {stage}",
        f"workload: {workload}",
        f"source_sha256: {source_digest(stage)}",
        f"dispatches_averaged: {n} (the driver's stage launches)",
        f"fetch_kib_per_dispatch: {f_kib:.1f}",
        f"write_kib_per_dispatch: {w_kib:.1f}",
        f"copy_256MiB_fetch_kib: {cf:.1f}",
        f"copy_256MiB_write_kib: {cw:.1f}",
        f"fetch_scale: {f_scale:.4f}",
        f"write_scale: {w_scale:.4f}",
        f"fetch_bytes_per_launch: {fetch_b:.0f}",
        f"write_bytes_per_launch: {write_b:.0f}",
        f"hbm_bytes_per_launch: {fetch_b + write_b:.0f}",
    ]
    return "\n".join(lines) + "\n"


def stats_summary(stats_csv: str, top: int, cmds: List[str]) -> str:
    rows = _rows(stats_csv)
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = ["# rocprofv3 kernel statistics", "", "commands (repo root; rocprofv3 run from /tmp "
           "with TMPDIR=/tmp):", *[f"  {c}" for c in cmds], "",
           f"{'calls':>7} {'avg_us':>9} {'min_us':>9} {'max_us':>9} {'total_ms':>9}  kernel"]
    for r in rows[:top]:
        out.append(f"{int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:9.2f} "
                   f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} "
                   f"{float(r['TotalDurationNs']) / 1e6:9.2f}  {short_name(r['Name'])}")
    return "\n".join(out) + "\n"


def load_traffic(stage: str, workload: str) -> Optional[dict]:
    """Bytes per launch recorded for `stage` on `workload`, or None when no
    summary exists or the kernel's sources changed since it was taken."""
    if stage not in KERNELS:
        return None
    path = os.path.join(PROFILES, f"{KERNELS[stage][0]}_{workload}_bytes.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            m = re.match(r"^([a-z0-9_]+): (.*)$", line.strip())
            if m:
                kv[m.group(1)] = m.group(2)
    if kv.get("source_sha256") != source_digest(stage):
        return None
    return {"bytes": float(kv["hbm_bytes_per_launch"]),
            "fetch_bytes": float(kv["fetch_bytes_per_launch"]),
            "write_bytes": float(kv["write_bytes_per_launch"]),
            "fetch_scale": float(kv["fetch_scale"]), "source": os.path.relpath(path, ROOT)}


def main(argv=None):
    ap = argparse.ArgumentParser()
    sp = ap.add_subparsers(dest="what", required=True)
    a = sp.add_parser("stats")
    a.add_argument("csv")
    a.add_argument("--top", type=int, default=20)
    a.add_argument("--cmd", action="append", default=[])
    b = sp.add_parser("bytes")
    b.add_argument("--fetch", required=True)
    b.add_argument("--write", required=True)
    b.add_argument("--stage", required=True, choices=sorted(KERNELS))
    b.add_argument("--workload", required=True)
    b.add_argument("--cmd", action="append", default=[])
    args = ap.parse_args(argv)
    if args.what == "stats":
        sys.stdout.write(stats_summary(args.csv, args.top, args.cmd))
    else:
        sys.stdout.write(bytes_summary(args.fetch, args.write, args.stage, args.workload,
                                       args.cmd))


if __name__ == "__main__":
    main()
