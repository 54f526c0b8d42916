"""Turns rocprofv3 outputs of `bench.py` into the short summaries kept under
`profiles/`, and reads the measured HBM traffic and MFMA activity back for the
benchmark.

    python -m paper_1412_7091_amd.profiling stats   TRACE_DIR OUT.md  "COMMAND"
    python -m paper_1412_7091_amd.profiling traffic FETCH_DIR WRITE_DIR OUT.txt "COMMANDS"
    python -m paper_1412_7091_amd.profiling mfma    PMC_DIR OUT.txt "COMMAND"
    python -m paper_1412_7091_amd.profiling tasks   CSV_TRACE_DIR BENCH_JSON OUT.md "COMMAND"

`mfma` reads one `--pmc SQ_INSTS_VALU_MFMA_MOPS_F32 SQ_VALU_MFMA_BUSY_CYCLES
GRBM_GUI_ACTIVE` run: per launch, the mean of each counter per dispatch, the
MFMA flops they imply (512 per MOP) and the busy fraction
SQ_VALU_MFMA_BUSY_CYCLES / ((GRBM_GUI_ACTIVE / 8 XCCs) x 256 CUs x 4 SIMDs).
`tasks` reads a CSV kernel trace of `bench.py --tasks` (every task of the step
launched alone) and names each step dispatch by its place in the step.

`stats` condenses a `--kernel-trace --stats` run into a Markdown table.
`traffic` reads two `--pmc` runs (FETCH_SIZE, then WRITE_SIZE; KiB per
dispatch) and scales each launch's counters by what the same counter read
for the benchmark's plain 64 MiB copy (the first copy dispatched after the
fill of its source), whose true traffic is known: 64 MiB read, 64 MiB
written.  Both read rocprofv3's database output (`*_results.db`).  The
result carries a digest of the kernel sources; `measured_traffic` returns
nothing once the sources change.
"""
from __future__ import annotations

import glob
import hashlib
import json
import os
import re
import sqlite3
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
REPO = os.path.dirname(PKG)
PROFILES = os.path.join(REPO, "profiles")
SOURCES = ["gemm_tile.h", "lst_internal.h", "step.hip", "lst_api.hip", "gemm.hip", "small.hip",
           "stabilize.hip", "online.hip", "lu.hip", "shifted.hip"]
CALIBRATION_BYTES = 64 << 20  # the benchmark's plain device-to-device copy


def source_digest() -> str:
    h = hashlib.sha256()
    for name in SOURCES:
        with open(os.path.join(PKG, "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def launch_of(kernel_name: str) -> str | None:
    """'launch1'..'launch5' for the step kernels (last template argument; 5 is the
    stabilisation's products), 'stab_fix_v' for the stabilisation's pass over V,
    else None."""
    m = re.search(r"step_kernel<[^<>]*?,\s*(\d)\s*>", kernel_name)
    if m:
        # 6 and 7 are launches 3 and 4 of a step that scatters its hot rows in launch 4
        return f"launch{ {'6': '3', '7': '4'}.get(m.group(1), m.group(1)) }"
    return "stab_fix_v" if "stab_fix_v_kernel" in kernel_name else None


def split_dispatches(rows) -> set:
    """Dispatch ids of step launches that ran one task alone (bench.py's split-task
    pass, lst_set_split_tasks): there a step kernel follows or precedes another
    dispatch of the same launch, which the default launch sequence never does.
    rows: (dispatch_id, kernel name) pairs."""
    steps = [(i, launch_of(n)) for i, n in sorted(rows)
             if (launch_of(n) or "").startswith("launch") and launch_of(n) != "launch5"]
    out = set()
    for j, (i, lk) in enumerate(steps):
        if (j > 0 and steps[j - 1][1] == lk) or (j + 1 < len(steps) and steps[j + 1][1] == lk):
            out.add(i)
    return out


def _db(directory: str) -> sqlite3.Connection:
    hits = sorted(glob.glob(os.path.join(directory, "**", "*_results.db"), recursive=True))
    if not hits:
        raise FileNotFoundError(f"no *_results.db under {directory}")
    return sqlite3.connect(hits[-1])


def per_launch_counter(directory: str, counter: str):
    """{launch or 'copy': mean counter value (KiB) per dispatch}."""
    con = _db(directory)
    rows = con.execute("select dispatch_id, kernel_name, value from counters_collection "
                       "where counter_name = ? order by dispatch_id", (counter,)).fetchall()
    split = split_dispatches([(i, n) for i, n, _ in rows])
    sums, counts = {}, {}
    fill_seen = False
    copy_val = None
    for i, name, val in rows:
        if i in split:
            continue
        key = launch_of(name)
        if key is not None:
            sums[key] = sums.get(key, 0.0) + float(val)
            counts[key] = counts.get(key, 0) + 1
        elif "FillFunctor" in name:
            fill_seen = True
        elif fill_seen and copy_val is None and re.search(r"copy", name, re.I):
            copy_val = float(val)
    out = {k: sums[k] / counts[k] for k in sums}
    if copy_val is not None:
        out["copy"] = copy_val
    return out


def write_traffic(fetch_dir: str, write_dir: str, out_path: str, commands: str) -> dict:
    fetch = per_launch_counter(fetch_dir, "FETCH_SIZE")
    write = per_launch_counter(write_dir, "WRITE_SIZE")
    if "copy" not in fetch or "copy" not in write:
        raise RuntimeError("calibration copy kernel not found in the counter runs")
    f_scale = fetch["copy"] * 1024.0 / CALIBRATION_BYTES  # counter bytes per true byte
    w_scale = write["copy"] * 1024.0 / CALIBRATION_BYTES
    launches = {}
    for k in sorted(set(fetch) | set(write)):
        if k == "copy":
            continue
        fb = fetch.get(k, 0.0) * 1024.0 / f_scale
        wb = write.get(k, 0.0) * 1024.0 / w_scale
        launches[k] = {"fetch_bytes": round(fb), "write_bytes": round(wb), "hbm_bytes": round(fb + wb)}
    res = {"source_digest": source_digest(), "fetch_scale": round(f_scale, 4),
           "write_scale": round(w_scale, 4), "copy_fetch_kib": fetch["copy"],
           "copy_write_kib": write["copy"], "launches": launches, "commands": commands}
    with open(out_path, "w") as f:
        f.write(json.dumps(res) + "\n")
    return res


def measured_traffic(workload: str) -> dict | None:
    """Per-launch HBM bytes from profiles/step_traffic_<workload>.txt, if current."""
    path = os.path.join(PROFILES, f"step_traffic_{workload}.txt")
    try:
        with open(path) as f:
            res = json.loads(f.read())
    except (OSError, ValueError):
        return None
    if res.get("source_digest") != source_digest():
        return None
    return res.get("launches")


def write_stats(trace_dir: str, out_path: str, command: str) -> None:
    con = _db(trace_dir)
    disp = con.execute("select dispatch_id, name, duration from kernels").fetchall()
    split = split_dispatches([(i, n) for i, n, _ in disp])
    groups = {}
    for i, name, dur in disp:
        groups.setdefault((name, i in split), []).append(float(dur))
    rows = sorted(((name + (" [one task per launch]" if sp else ""), len(v), sum(v),
                    sum(v) / len(v), min(v), max(v)) for (name, sp), v in groups.items()),
                  key=lambda r: -r[2])
    total = sum(r[2] for r in rows) or 1.0
    lines = ["# Kernel time summary (rocprofv3 --kernel-trace --stats)", "",
             f"Command: `{command}`", "",
             "Durations are per dispatch, kernel execution only (ns from the trace, shown in us).", "",
             "| Kernel | Launch | Calls | Total (us) | Average (us) | Min (us) | Max (us) | Share |",
             "|---|---|---|---|---|---|---|---|"]
    for name, calls, tot, avg, mn, mx in rows:
        short = name if len(name) < 90 else name[:60] + "..." + name[-27:]
        lines.append(f"| `{short}` | {launch_of(name) or ''} | {calls} | {tot / 1e3:.1f} | "
                     f"{avg / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} | {100 * tot / total:.1f}% |")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")


MFMA_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_F32", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
N_CU, SIMD_PER_CU = 256, 4
N_XCC = 8          # GRBM_GUI_ACTIVE has one instance per XCC; the database sums them
FLOPS_PER_MOP = 512
CLOCK_GHZ = 2.4


def write_mfma(pmc_dir: str, out_path: str, command: str) -> dict:
    vals = {c: per_launch_counter(pmc_dir, c) for c in MFMA_COUNTERS}
    launches = {}
    for k in sorted(vals["GRBM_GUI_ACTIVE"]):
        if k == "copy":
            continue
        mops = vals["SQ_INSTS_VALU_MFMA_MOPS_F32"].get(k, 0.0)
        busy = vals["SQ_VALU_MFMA_BUSY_CYCLES"].get(k, 0.0)
        gui = vals["GRBM_GUI_ACTIVE"][k]
        cycles = gui / N_XCC
        launches[k] = {"mops_f32": mops, "mfma_busy_cycles": busy, "gui_active": gui,
                       "active_us_at_2p4GHz": round(cycles / (CLOCK_GHZ * 1e3), 3),
                       "mfma_flops": FLOPS_PER_MOP * mops,
                       "busy_frac": round(busy / (cycles * N_CU * SIMD_PER_CU), 5) if gui else None}
    res = {"source_digest": source_digest(), "launches": launches, "command": command,
           "busy_frac_definition": "SQ_VALU_MFMA_BUSY_CYCLES / ((GRBM_GUI_ACTIVE / 8) * 256 * 4): "
                                   "MFMA-busy SIMD cycles over the SIMD cycles of the dispatch"}
    with open(out_path, "w") as f:
        f.write(json.dumps(res) + "\n")
    return res


def measured_mfma(workload: str) -> dict | None:
    """Per-launch MFMA counters from profiles/step_mfma_<workload>.txt, if current."""
    path = os.path.join(PROFILES, f"step_mfma_{workload}.txt")
    try:
        with open(path) as f:
            res = json.loads(f.read())
    except (OSError, ValueError):
        return None
    if res.get("source_digest") != source_digest():
        return None
    return res.get("launches")


def split_order(m: int) -> dict:
    """Task order of each step kernel (by launch number) when every task runs alone."""
    l2 = ["gemm", "solve", "yy", "scalars"] if m <= 128 else ["solve", "yy", "gemm", "scalars"]
    return {"launch1": ["gemm", "targets"], "launch2": l2, "launch3": ["scatter", "gemm"],
            "launch4": ["gemm", "clear"]}


def write_tasks(trace_dir: str, bench_json: str, out_path: str, command: str) -> dict:
    import csv

    with open(bench_json) as f:
        line = [ln for ln in f if ln.strip().startswith("{")][-1]
    bench = json.loads(line)
    m = bench["config"]["m"]
    order = split_order(m)
    hits = sorted(glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True))
    if not hits:
        raise FileNotFoundError(f"no kernel_trace.csv under {trace_dir}")
    with open(hits[-1]) as f:
        rows = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
    seen, durs = {}, {}
    for r in rows:
        lk = launch_of(r["Kernel_Name"])
        if lk is None or lk == "stab_fix_v":
            continue
        if lk not in order:
            continue
        i = seen.get(lk, 0)
        seen[lk] = i + 1
        name = f"{lk}.{order[lk][i % len(order[lk])]}"
        durs.setdefault(name, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    import statistics

    lines = ["# Step tasks launched alone (rocprofv3 kernel trace of `bench.py --tasks`)", "",
             f"Command: `{command}`", "",
             f"Workload {bench['config']['workload']}: D = {bench['config']['D']}, "
             f"d = {bench['config']['d']}, m = {m}, K = {bench['config']['K']}; "
             f"{bench['distinct_rows']} distinct target rows in the last step.", "",
             "| Task | Dispatches | Median (us) | Mean (us) |",
             "|---|---|---|---|"]
    summary = {}
    for name in sorted(durs):
        v = durs[name]
        summary[name] = {"median_us": round(statistics.median(v), 3),
                         "mean_us": round(statistics.fmean(v), 3)}
        lines.append(f"| {name} | {len(v)} | {statistics.median(v):.2f} | "
                     f"{statistics.fmean(v):.2f} |")
    lines += ["", "| Part | Tasks | Algorithmic bytes | Median (us) | GB/s | of 8 TB/s |",
              "|---|---|---|---|---|---|"]
    for part in ("gather", "scatter"):
        b = bench["tasks"].get(part)
        if not b:
            continue
        t = sum(summary[p]["median_us"] for p in b["tasks"] if p in summary)
        gbs = b["bytes"] / (t * 1e-6) / 1e9 if t else 0.0
        summary[part] = {"bytes": b["bytes"], "median_us": round(t, 3), "hbm_gbs": round(gbs, 1),
                         "hbm_frac": round(gbs / 8000.0, 4)}
        lines.append(f"| {part} | {' + '.join(b['tasks'])} | {b['bytes']:.0f} | {t:.2f} | "
                     f"{gbs:.0f} | {100 * gbs / 8000.0:.1f}% |")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    return summary


def main(argv):
    if len(argv) >= 4 and argv[0] == "stats":
        write_stats(argv[1], argv[2], argv[3])
    elif len(argv) >= 5 and argv[0] == "traffic":
        print(json.dumps(write_traffic(argv[1], argv[2], argv[3], argv[4])))
    elif len(argv) >= 4 and argv[0] == "mfma":
        print(json.dumps(write_mfma(argv[1], argv[2], argv[3])))
    elif len(argv) >= 5 and argv[0] == "tasks":
        print(json.dumps(write_tasks(argv[1], argv[2], argv[3], argv[4])))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
