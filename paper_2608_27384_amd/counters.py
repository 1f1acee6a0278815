"""Summaries of rocprofv3 output for the measurement record (no GPU work).

* ``stats``: the per-kernel table of ``rocprofv3 --kernel-trace --stats
  --output-format csv`` (``*_kernel_stats.csv``), shortened to the kernels
  that matter, as text.
* ``trace``: per-kernel durations from the same run's ``*_kernel_trace.csv``,
  split into the decode steps and the stage timing that follows them.
* ``bytes``: HBM bytes per launch of one kernel, from two counter runs of
  ``bench.py --pmc-driver STAGES``: one with ``--pmc FETCH_SIZE``, one with
  ``--pmc WRITE_SIZE`` (``*_counter_collection.csv``, KiB per dispatch).
* ``step-bytes``: HBM bytes per decode step (every kernel of the step), from
  the same two counter runs of ``bench.py --pmc-driver step``.
* ``step-mfma``: MFMA work and utilisation per decode step and per kernel,
  from one run of ``bench.py --pmc-driver step`` with ``--pmc
  SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 GRBM_GUI_ACTIVE``.

Byte counters are scaled by what they read for passes of known size that
the driver makes after the measured kernels: a 256 MiB device copy, a 256
MiB read-only sum and a 256 MiB write-only fill.  The copy sets the scale;
the sum (reads) and the fill (writes) are a second, independent calibration
and both factors are recorded.  Every summary records a digest of the
sources it depends on, so that a reader (bench.py) can tell when the kernels
have changed since the counters were taken.

python -m paper_2608_27384_amd.counters stats CSV [--top N] [--cmd TEXT]
python -m paper_2608_27384_amd.counters bytes --fetch CSV --write CSV --kernel KEY
       --workload NAME --launches N [--cmd TEXT ...]
python -m paper_2608_27384_amd.counters step-bytes --fetch CSV --write CSV --workload NAME
python -m paper_2608_27384_amd.counters step-mfma --csv CSV --workload NAME
python -m paper_2608_27384_amd.counters trace KERNEL_TRACE_CSV --workload NAME
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import re
import sys
from collections import OrderedDict
from typing import Dict, List, Optional, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
PROFILES = os.path.join(ROOT, "profiles")

CAL_BYTES = 256 << 20           # size of each calibration pass
SIMD_NUM = 1024                 # 256 CUs x 4 SIMDs
XCD_NUM = 8                     # GRBM_GUI_ACTIVE arrives summed over the 8 dies

GEMM_SRC = ("csrc/fv_gemm.hip", "csrc/fv_internal.h")
ATTN_SRC = ("csrc/fv_attn.hip", "csrc/fv_internal.h")
MISC_SRC = ("csrc/fv_misc.hip", "csrc/fv_internal.h")
ALL_SRC = ("csrc/fv_gemm.hip", "csrc/fv_attn.hip", "csrc/fv_misc.hip", "csrc/fv_runtime.hip",
           "csrc/fv_internal.h")

# kernel key (substring of its name in a trace) -> source files that define it
KERNELS: Dict[str, Tuple[str, ...]] = {
    "EpiBiasF32": GEMM_SRC, "EpiQkv": GEMM_SRC, "EpiGeglu": GEMM_SRC, "EpiGelu": GEMM_SRC,
    "EpiNone": GEMM_SRC, "EpiGatedResid": GEMM_SRC,
    "attn16d_kernel": ATTN_SRC, "attn16_kernel": ATTN_SRC, "attn_kernel": ATTN_SRC,
    "attn_combine": ATTN_SRC,
    "resid_norm_kernel": MISC_SRC, "adarms_kernel": MISC_SRC,
}


def short_name(name: str) -> str:
    name = re.sub(r"fv::\(anonymous namespace\)::", "", name)
    name = re.sub(r"fv::", "", name)
    return re.sub(r"\(.*", "", name)


def digest(files) -> str:
    h = hashlib.sha256()
    for rel in files:
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _rows(path: str) -> List[dict]:
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def dispatches(path: str) -> List[Tuple[str, Dict[str, float]]]:
    """[(kernel name, {counter: value})] in dispatch order.  Several rows of
    one (dispatch, counter) are combined: summed, except GRBM_* (maximum)."""
    rows = _rows(path)
    idk = "Dispatch_Id" if rows and "Dispatch_Id" in rows[0] else "Correlation_Id"
    out: "OrderedDict[int, Tuple[str, Dict[str, float]]]" = OrderedDict()
    for r in sorted(rows, key=lambda r: int(r[idk])):
        d = int(r[idk])
        name, vals = out.setdefault(d, (r["Kernel_Name"], {}))
        c, v = r["Counter_Name"], float(r["Counter_Value"])
        if c in vals:
            vals[c] = max(vals[c], v) if c.startswith("GRBM") else vals[c] + v
        else:
            vals[c] = v
    return list(out.values())


def _calibration(ds, counter: str) -> Dict[str, float]:
    """KiB the counter reads for each 256 MiB calibration pass: the largest
    reading among the dispatches of the pass's kernel (other, small
    dispatches of the same kernels happen during set-up).  The library's own
    kernels never count, whatever their names (its prefix install is a large
    "copy" kernel)."""
    def big(pred):
        vals = [v.get(counter, 0.0) for n, v in ds if pred(n) and "fv::" not in n]
        return max(vals) if vals else None
    return {"copy": big(lambda n: "copyBuffer" in n or "copy_kernel" in n),
            "sum": big(lambda n: "reduce_kernel" in n),
            "fill": big(lambda n: "FillFunctor" in n)}


def _scale(cal: Dict[str, Optional[float]], which: str) -> float:
    kib = cal.get(which)
    if not kib:
        raise ValueError(f"no {which} calibration dispatch")
    return CAL_BYTES / (kib * 1024.0)


def _cal_lines(fc, wc) -> List[str]:
    def f(x):
        return "none" if x is None else f"{x:.1f}"
    lines = [f"calibration_fetch_kib: copy {f(fc['copy'])}, sum {f(fc['sum'])}, "
             f"fill {f(fc['fill'])} (256 MiB each)",
             f"calibration_write_kib: copy {f(wc['copy'])}, sum {f(wc['sum'])}, "
             f"fill {f(wc['fill'])}"]
    fs = [CAL_BYTES / (fc[k] * 1024.0) for k in ("copy", "sum") if fc.get(k)]
    ws = [CAL_BYTES / (wc[k] * 1024.0) for k in ("copy", "fill") if wc.get(k)]
    lines.append("fetch_scale_copy_sum: " + " ".join(f"{x:.4f}" for x in fs))
    lines.append("write_scale_copy_fill: " + " ".join(f"{x:.4f}" for x in ws))
    return lines


def bytes_summary(fetch_csv, write_csv, kernel, workload, launches, cmds) -> str:
    fd, wd = dispatches(fetch_csv), dispatches(write_csv)
    fmine = [v["FETCH_SIZE"] for n, v in fd if kernel in n]
    wmine = [v["WRITE_SIZE"] for n, v in wd if kernel in n]
    if len(fmine) < launches or len(wmine) < launches:
        raise ValueError(f"{len(fmine)}/{len(wmine)} dispatches of *{kernel}* (want {launches})")
    f_kib = sum(fmine[-launches:]) / launches
    w_kib = sum(wmine[-launches:]) / launches
    fc, wc = _calibration(fd, "FETCH_SIZE"), _calibration(wd, "WRITE_SIZE")
    fs, ws = _scale(fc, "copy"), _scale(wc, "copy")
    fetch_b, write_b = f_kib * 1024.0 * fs, w_kib * 1024.0 * ws
    lines = [
        f"# HBM bytes per launch: {kernel}, workload {workload}",
        "",
        "commands (repo root; rocprofv3 run from /tmp with TMPDIR=/tmp):",
        *[f"  {c}" for c in cmds],
        "",
        f"kernel_match: {kernel}",
        f"workload: {workload}",
        f"source_sha256: {digest(KERNELS[kernel])}",
        f"dispatches_averaged: {launches} (the driver's stage launches)",
        f"fetch_kib_per_dispatch: {f_kib:.1f}",
        f"write_kib_per_dispatch: {w_kib:.1f}",
        *_cal_lines(fc, wc),
        f"fetch_scale: {fs:.4f}",
        f"write_scale: {ws:.4f}",
        f"fetch_bytes_per_launch: {fetch_b:.0f}",
        f"write_bytes_per_launch: {write_b:.0f}",
        f"hbm_bytes_per_launch: {fetch_b + write_b:.0f}",
    ]
    return "\n".join(lines) + "\n"


def _step_end(name: str) -> bool:
    """A decode step ends with its Euler update: the Euler kernel, or the
    velocity head with the update fused in."""
    return "euler_shift_kernel" in name or "final_small_kernel<true>" in name


def _step_window(ds) -> Tuple[int, int, int]:
    """(first, last, steps): the dispatches after the first decode step
    (warm-up) up to the end of the last one; a step ends with its Euler
    update."""
    ends = [i for i, (n, _) in enumerate(ds) if _step_end(n)]
    if len(ends) < 2:
        raise ValueError("need a warm-up step and at least one measured step")
    return ends[0] + 1, ends[-1], len(ends) - 1


def step_bytes_summary(fetch_csv, write_csv, workload, cmds) -> str:
    fd, wd = dispatches(fetch_csv), dispatches(write_csv)
    a, b, n = _step_window(fd)
    a2, b2, n2 = _step_window(wd)
    f_kib = sum(v.get("FETCH_SIZE", 0.0) for _, v in fd[a:b + 1]) / n
    w_kib = sum(v.get("WRITE_SIZE", 0.0) for _, v in wd[a2:b2 + 1]) / n2
    fc, wc = _calibration(fd, "FETCH_SIZE"), _calibration(wd, "WRITE_SIZE")
    fs, ws = _scale(fc, "copy"), _scale(wc, "copy")
    per_kernel: Dict[str, float] = {}
    for name, v in fd[a:b + 1]:
        per_kernel[short_name(name)] = per_kernel.get(short_name(name), 0.0) + \
            v.get("FETCH_SIZE", 0.0) * 1024.0 * fs / n
    for name, v in wd[a2:b2 + 1]:
        per_kernel[short_name(name)] = per_kernel.get(short_name(name), 0.0) + \
            v.get("WRITE_SIZE", 0.0) * 1024.0 * ws / n2
    lines = [
        f"# HBM bytes per decode step (all kernels), workload {workload}",
        "",
        "commands (repo root; rocprofv3 run from /tmp with TMPDIR=/tmp):",
        *[f"  {c}" for c in cmds],
        "",
        f"workload: {workload}",
        f"source_sha256: {digest(ALL_SRC)}",
        f"steps_summed: {n} (after one warm-up step)",
        f"dispatches_per_step: {(b - a + 1) / n:.1f}",
        *_cal_lines(fc, wc),
        f"fetch_scale: {fs:.4f}",
        f"write_scale: {ws:.4f}",
        f"fetch_bytes_per_step: {f_kib * 1024.0 * fs:.0f}",
        f"write_bytes_per_step: {w_kib * 1024.0 * ws:.0f}",
        f"hbm_bytes_per_step: {f_kib * 1024.0 * fs + w_kib * 1024.0 * ws:.0f}",
        "",
        "HBM bytes per step by kernel (fetch + write, scaled):",
    ]
    for k, v in sorted(per_kernel.items(), key=lambda kv: -kv[1])[:16]:
        lines.append(f"  {v / 1e6:10.2f} MB  {k}")
    return "\n".join(lines) + "\n"


def step_mfma_summary(csv_path, workload, cmds) -> str:
    ds = dispatches(csv_path)
    a, b, n = _step_window(ds)
    busy = mops = gui = 0.0
    per: Dict[str, List[float]] = {}
    for name, v in ds[a:b + 1]:
        bsy = v.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        mo = v.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0)
        g = v.get("GRBM_GUI_ACTIVE", 0.0)
        busy, mops, gui = busy + bsy, mops + mo, gui + g
        p = per.setdefault(short_name(name), [0.0, 0.0, 0.0])
        p[0] += bsy
        p[1] += mo
        p[2] += g
    lines = [
        f"# MFMA work and utilisation per decode step, workload {workload}",
        "",
        "commands (repo root; rocprofv3 run from /tmp with TMPDIR=/tmp):",
        *[f"  {c}" for c in cmds],
        "",
        f"workload: {workload}",
        f"source_sha256: {digest(ALL_SRC)}",
        f"steps_summed: {n} (after one warm-up step)",
        f"mfma_busy_cycles_per_step: {busy / n:.0f}",
        f"gui_active_cycles_per_step: {gui / XCD_NUM / n:.0f}",
        f"mfma_bf16_flops_per_step: {mops * 512.0 / n:.0f}",
        f"mfma_util_step: {busy / (gui / XCD_NUM * SIMD_NUM):.4f}",
        "  (sum over the step's dispatches of SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE of one die"
        " x 1024 SIMDs), rocprofv3's MfmaUtil formula; the counter run reports GRBM_GUI_ACTIVE"
        " summed over the 8 dies, hence / 8; each dispatch runs alone under counters)",
        "",
        "per kernel: mfma_util, bf16 MFMA GFLOP per step, share of busy cycles",
    ]
    for k, (bs, mo, g) in sorted(per.items(), key=lambda kv: -kv[1][0])[:12]:
        util = bs / (g / XCD_NUM * SIMD_NUM) if g else 0.0
        lines.append(f"  {util:7.4f} {mo * 512.0 / n / 1e9:10.2f} {bs / busy if busy else 0:6.3f}  {k}")
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


def _kernel_table(rows: List[Tuple[str, float]]) -> List[str]:
    """[(kernel, microseconds)] -> per-kernel lines, largest total first."""
    agg: Dict[str, List[float]] = {}
    for name, us in rows:
        agg.setdefault(short_name(name), []).append(us)
    out = [f"{'calls':>7} {'avg_us':>9} {'min_us':>9} {'max_us':>9} {'total_ms':>9}  kernel"]
    for k, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"{len(v):7d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f} "
                   f"{sum(v) / 1e3:9.2f}  {k}")
    return out


def trace_summary(trace_csv: str, workload: str, cmds: List[str]) -> str:
    """Kernel durations of a bench.py run, in two windows: the decode steps
    (from the first time-embedding kernel to the last Euler update) and the
    stage timing that follows them (one kernel replayed in a graph, layers
    cycling)."""
    rows = _rows(trace_csv)
    ev = sorted(((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"])
                 for r in rows), key=lambda x: x[0])
    first = next(i for i, e in enumerate(ev) if "time_embed_kernel" in e[2])
    last = max(i for i, e in enumerate(ev) if _step_end(e[2]))
    steps = sum(1 for e in ev[first:last + 1] if _step_end(e[2]))
    span_us = (ev[last][1] - ev[first][0]) / 1e3
    in_step = [(n, (b - a) / 1e3) for a, b, n in ev[first:last + 1]]
    after = [(n, (b - a) / 1e3) for a, b, n in ev[last + 1:]]
    busy = sum(us for _, us in in_step)
    lines = ["# rocprofv3 kernel trace: decode steps, then the stage timing", "",
             "commands (repo root; rocprofv3 run from /tmp with TMPDIR=/tmp):",
             *[f"  {c}" for c in cmds], "",
             f"workload: {workload}",
             f"source_sha256: {digest(ALL_SRC)}",
             f"steps: {steps}",
             f"step_span_us: {span_us / steps:.1f} (first to last kernel of the steps, per step)",
             f"kernel_busy_us_per_step: {busy / steps:.1f}",
             f"dispatches_per_step: {len(in_step) / steps:.1f}",
             "",
             "decode steps (graph replays; warm-up and timed steps):"]
    lines += _kernel_table(in_step)
    lines += ["", "stage timing after the steps (fv_debug_stage: one kernel per graph, "
              "layers cycling):"]
    lines += _kernel_table(after)
    return "\n".join(lines) + "\n"


def load_in_step(workload: str) -> Optional[dict]:
    """Per-kernel in-step average durations from the committed trace summary."""
    path = os.path.join(PROFILES, f"{workload}_kernel_trace.txt")
    if not os.path.exists(path):
        return None
    kv, table, sect = {}, {}, None
    with open(path) as f:
        for line in f:
            m = re.match(r"^([a-z0-9_]+): (.*)$", line.strip())
            if m:
                kv[m.group(1)] = m.group(2)
            if line.startswith("decode steps"):
                sect = "step"
            elif line.startswith("stage timing"):
                sect = None
            m2 = re.match(r"^\s*(\d+)\s+([\d.]+)\s+[\d.]+\s+[\d.]+\s+[\d.]+\s+(.*)$", line)
            if sect == "step" and m2:
                table[m2.group(3).strip()] = float(m2.group(2))
    if not table:
        return None
    return {"avg_us": table, "current": kv.get("source_sha256") == digest(ALL_SRC),
            "source": os.path.relpath(path, ROOT)}


def _kv(path: str) -> Dict[str, str]:
    kv = {}
    with open(path) as f:
        for line in f:
            m = re.match(r"^([a-z0-9_]+): (.*)$", line.strip())
            if m:
                kv[m.group(1)] = m.group(2)
    return kv


def load_traffic(kernel: str, workload: str) -> Optional[dict]:
    """Bytes per launch recorded for `kernel` on `workload`, or None when no
    summary exists or the kernel's sources changed since it was taken."""
    if kernel not in KERNELS:
        return None
    path = os.path.join(PROFILES, f"{kernel}_{workload}_bytes.txt")
    if not os.path.exists(path):
        return None
    kv = _kv(path)
    if kv.get("source_sha256") != digest(KERNELS[kernel]):
        return None
    return {"bytes": float(kv["hbm_bytes_per_launch"]),
            "fetch_bytes": float(kv["fetch_bytes_per_launch"]),
            "write_bytes": float(kv["write_bytes_per_launch"]),
            "fetch_scale": float(kv["fetch_scale"]), "source": os.path.relpath(path, ROOT)}


def load_step_bytes(workload: str) -> Optional[dict]:
    path = os.path.join(PROFILES, f"{workload}_step_bytes.txt")
    if not os.path.exists(path):
        return None
    kv = _kv(path)
    return {"hbm_bytes_per_step": float(kv["hbm_bytes_per_step"]),
            "fetch_bytes_per_step": float(kv["fetch_bytes_per_step"]),
            "write_bytes_per_step": float(kv["write_bytes_per_step"]),
            "current": kv.get("source_sha256") == digest(ALL_SRC),
            "source": os.path.relpath(path, ROOT)}


def load_step_mfma(workload: str) -> Optional[dict]:
    path = os.path.join(PROFILES, f"{workload}_step_mfma.txt")
    if not os.path.exists(path):
        return None
    kv = _kv(path)
    return {"mfma_util": float(kv["mfma_util_step"]),
            "mfma_bf16_flops_per_step": float(kv["mfma_bf16_flops_per_step"]),
            "current": kv.get("source_sha256") == digest(ALL_SRC),
            "source": os.path.relpath(path, ROOT)}


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
    b.add_argument("--kernel", required=True, choices=sorted(KERNELS))
    b.add_argument("--workload", required=True)
    b.add_argument("--launches", type=int, default=20)
    b.add_argument("--cmd", action="append", default=[])
    c = sp.add_parser("step-bytes")
    c.add_argument("--fetch", required=True)
    c.add_argument("--write", required=True)
    c.add_argument("--workload", required=True)
    c.add_argument("--cmd", action="append", default=[])
    t = sp.add_parser("trace")
    t.add_argument("csv")
    t.add_argument("--workload", required=True)
    t.add_argument("--cmd", action="append", default=[])
    d = sp.add_parser("step-mfma")
    d.add_argument("--csv", required=True)
    d.add_argument("--workload", required=True)
    d.add_argument("--cmd", action="append", default=[])
    args = ap.parse_args(argv)
    if args.what == "stats":
        sys.stdout.write(stats_summary(args.csv, args.top, args.cmd))
    elif args.what == "bytes":
        sys.stdout.write(bytes_summary(args.fetch, args.write, args.kernel, args.workload,
                                       args.launches, args.cmd))
    elif args.what == "trace":
        sys.stdout.write(trace_summary(args.csv, args.workload, args.cmd))
    elif args.what == "step-bytes":
        sys.stdout.write(step_bytes_summary(args.fetch, args.write, args.workload, args.cmd))
    else:
        sys.stdout.write(step_mfma_summary(args.csv, args.workload, args.cmd))


if __name__ == "__main__":
    main()
