"""Summaries of rocprofv3 output for this library's kernels.

    python -m paper_2609_12399_amd.rocprof_summary trace <dir-or-file>
    python -m paper_2609_12399_amd.rocprof_summary pmc <FETCH_SIZE dir> <WRITE_SIZE dir>
    python -m paper_2609_12399_amd.rocprof_summary mfma <counter dir> [<trace dir>]
    python -m paper_2609_12399_amd.rocprof_summary counters <kernel-substring> <dir> [<dir> ...]

``trace`` reads a ``--kernel-trace`` result (``*_kernel_trace.csv`` or a
``*_results.db``) and prints one markdown row per kernel instance (calls,
average / median / min duration).  ``pmc`` reads two ``--pmc FETCH_SIZE`` and
``--pmc WRITE_SIZE`` runs (``*_counter_collection.csv``) and prints the
average KiB per dispatch of each counter and kernel, raw and scaled by the
factors a plain copy of known size gives (the largest device copy in the
same runs, whose true read and write sizes equal its byte count).  ``mfma``
reads a ``--pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES
GRBM_GUI_ACTIVE`` run and prints, per kernel, the bf16 MFMA flops per dispatch
(MOPS x 512), the matrix-core busy fraction (busy cycles over active cycles
times the 1024 SIMDs, rocprofv3's MfmaUtil; the CSV sums GRBM_GUI_ACTIVE over
the 8 XCDs, so one XCD's active cycles are taken as that sum / 8) and, given a
kernel trace of the same command, the achieved bf16 MFMA rate.  ``counters``
reads any number of ``--pmc`` runs and prints, for every kernel whose short
name contains the substring, the average per dispatch of each counter found.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import os
import re
import sqlite3
import statistics
import sys
from collections import defaultdict

DECODE_RE = re.compile(r"decode_kernel<(\d+), (\d+), (\d+), (\d+), (\d+), (true|false), "
                       r"(true|false)(?:, (true|false))?>")


def short_name(name: str) -> str:
    m = DECODE_RE.search(name)
    if m:
        dk, dv, mb, nblk, chain, bf16, fused, borrow = m.groups()
        mode = "fused" if fused == "true" else "decode"
        records = "" if borrow is None else (", borrowed" if borrow == "true" else ", arena")
        return (f"decode_kernel<{mode}, d={dk}, chain={chain}, "
                f"{'bf16' if bf16 == 'true' else 'f32'}{records}>")
    for k in ("resolve_kernel", "append_kernel", "prefill_kernel", "prefill_chunk_kernel",
              "prefill_scan_kernel", "fullstate_kernel", "clear_status_kernel"):
        if k in name:
            return k
    m = re.search(r"(select_\w+_kernel)(<[^>]*>)?", name)
    if m:
        return m.group(1) + (m.group(2) or "")
    name = re.sub(r"\(.*", "", name).replace("void ", "")
    return name[:60]


def source_sha256(path: str) -> str:
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def _find(path: str, pattern: str) -> list:
    if os.path.isfile(path):
        return [path]
    return sorted(glob.glob(os.path.join(path, "**", pattern), recursive=True))


def trace_rows(path: str):
    """(name, grid, workgroup, duration_ns) per dispatch."""
    csvs = _find(path, "*kernel_trace.csv")
    if csvs:
        for f in csvs:
            for r in csv.DictReader(open(f)):
                dur = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
                yield (r["Kernel_Name"], int(r.get("Grid_Size_X", r.get("Grid_Size", 0))),
                       int(r.get("Workgroup_Size_X", r.get("Workgroup_Size", 0))), dur)
        return
    for f in _find(path, "*results.db"):
        db = sqlite3.connect(f)
        for name, dur, gx, wx in db.execute(
                "select name, duration, grid_x, workgroup_x from kernels order by start"):
            yield name, gx, wx, dur


def summarize_trace(path: str) -> str:
    d = defaultdict(list)
    for name, grid, wg, dur in trace_rows(path):
        d[(short_name(name), grid // max(wg, 1), wg)].append(dur / 1e3)
    out = ["| kernel | workgroups | threads | calls | avg us | median us | min us |",
           "|---|---|---|---|---|---|---|"]
    for (name, g, w), v in sorted(d.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| {name} | {g} | {w} | {len(v)} | {sum(v) / len(v):.2f} | "
                   f"{statistics.median(v):.2f} | {min(v):.2f} |")
    return "\n".join(out)


def pmc_rows(path: str):
    for f in _find(path, "*counter_collection.csv"):
        for r in csv.DictReader(open(f)):
            yield r["Kernel_Name"], int(r["Grid_Size"]), int(r["Workgroup_Size"]), \
                r["Counter_Name"], float(r["Counter_Value"])


def copy_calibration(rows) -> float:
    """Bytes-per-KiB-reported factor from the largest device copy dispatch."""
    best = None
    for name, grid, wg, cname, val in rows:
        if "copyBuffer" in name and (best is None or val > best):
            best = val
    return best


def summarize_pmc(fetch_dir: str, write_dir: str, copy_bytes: int | None = None) -> str:
    frows = list(pmc_rows(fetch_dir))
    wrows = list(pmc_rows(write_dir))
    fmax, wmax = copy_calibration(frows), copy_calibration(wrows)
    # the largest copy reads and writes the same number of bytes; WRITE_SIZE
    # of a copy counts exactly its size, so it calibrates FETCH_SIZE too
    kib = copy_bytes / 1024 if copy_bytes else wmax
    ff, wf = kib / fmax, kib / wmax
    out = [f"calibration: largest device copy = {kib:.0f} KiB read and written; "
           f"FETCH_SIZE reads {fmax:.1f} KiB (factor {ff:.4f}), "
           f"WRITE_SIZE reads {wmax:.1f} KiB (factor {wf:.4f})", "",
           "| kernel | workgroups | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | "
           "read MB (scaled) | written MB (scaled) | total MB |",
           "|---|---|---|---|---|---|---|---|"]
    acc = defaultdict(lambda: [[], []])
    for rows, i in ((frows, 0), (wrows, 1)):
        for name, grid, wg, cname, val in rows:
            acc[(short_name(name), grid // max(wg, 1))][i].append(val)
    for (name, g), (fv, wv) in sorted(acc.items(), key=lambda kv: -sum(kv[1][0])):
        if not fv or not wv:
            continue
        f, w = sum(fv) / len(fv), sum(wv) / len(wv)
        rd, wr = f * ff * 1024 / 1e6, w * wf * 1024 / 1e6
        out.append(f"| {name} | {g} | {len(fv)} | {f:.1f} | {w:.1f} | {rd:.2f} | {wr:.2f} | "
                   f"{rd + wr:.2f} |")
    return "\n".join(out)


SIMD_NUM = 1024  # MI355X: 256 CUs x 4 SIMDs
XCD_NUM = 8


def mfma_stats(counter_dir: str):
    """{(kernel, workgroups): (dispatches, flops, busy cycles, active cycles)},
    averages per dispatch."""
    acc = defaultdict(lambda: defaultdict(list))
    for name, grid, wg, cname, val in pmc_rows(counter_dir):
        acc[(short_name(name), grid // max(wg, 1))][cname].append(val)
    out = {}
    for key, c in acc.items():
        mops = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", [])
        busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", [])
        gui = c.get("GRBM_GUI_ACTIVE", [])
        if not (mops and busy and gui):
            continue
        avg = lambda v: sum(v) / len(v)
        out[key] = (len(mops), avg(mops) * 512, avg(busy), avg(gui))
    return out


def mfma_util(busy: float, gui_sum: float) -> float:
    """Per cent of SIMD cycles with the matrix core busy."""
    return 100.0 * busy / (gui_sum / XCD_NUM * SIMD_NUM)


def summarize_mfma(counter_dir: str, trace_dir: str | None = None) -> str:
    durs = defaultdict(list)
    if trace_dir:
        for name, grid, wg, dur in trace_rows(trace_dir):
            durs[(short_name(name), grid // max(wg, 1))].append(dur)
    out = ["| kernel | workgroups | dispatches | bf16 MFMA GFLOP | MfmaUtil % | "
           "avg us (trace) | bf16 MFMA TFLOP/s |",
           "|---|---|---|---|---|---|---|"]
    for (name, g), (n, flops, busy, gui) in sorted(mfma_stats(counter_dir).items(),
                                                    key=lambda kv: -kv[1][1]):
        if flops == 0:
            continue
        util = mfma_util(busy, gui)
        d = durs.get((name, g))
        us = sum(d) / len(d) / 1e3 if d else None
        rate = f"{flops / (us * 1e-6) / 1e12:.1f}" if us else "-"
        out.append(f"| {name} | {g} | {n} | {flops / 1e9:.3f} | {util:.2f} | "
                   f"{'-' if us is None else f'{us:.2f}'} | {rate} |")
    return "\n".join(out)


def summarize_counters(sub: str, dirs) -> str:
    acc = defaultdict(lambda: defaultdict(list))
    names = []
    for d in dirs:
        for name, grid, wg, cname, val in pmc_rows(d):
            k = short_name(name)
            if sub not in k:
                continue
            acc[(k, grid // max(wg, 1))][cname].append(val)
            if cname not in names:
                names.append(cname)
    out = ["| kernel | workgroups | " + " | ".join(names) + " |",
           "|---|---|" + "---|" * len(names)]
    for (k, g), c in sorted(acc.items()):
        vals = [f"{sum(c[n]) / len(c[n]):.4g}" if c.get(n) else "-" for n in names]
        out.append(f"| {k} | {g} | " + " | ".join(vals) + " |")
    return "\n".join(out)


if __name__ == "__main__":
    if len(sys.argv) >= 3 and sys.argv[1] == "trace":
        print(summarize_trace(sys.argv[2]))
    elif len(sys.argv) >= 4 and sys.argv[1] == "pmc":
        print(summarize_pmc(sys.argv[2], sys.argv[3]))
    elif len(sys.argv) >= 4 and sys.argv[1] == "counters":
        print(summarize_counters(sys.argv[2], sys.argv[3:]))
    elif len(sys.argv) >= 3 and sys.argv[1] == "mfma":
        print(summarize_mfma(sys.argv[2], sys.argv[3] if len(sys.argv) > 3 else None))
    else:
        print(__doc__)
        sys.exit(2)
