"""Turns rocprofv3 outputs of `bench.py` into the short summaries kept under
`profiles/`, and reads the measured HBM traffic back for the benchmark.

    python -m paper_1412_7091_amd.profiling stats   TRACE_DIR OUT.md  "COMMAND"
    python -m paper_1412_7091_amd.profiling traffic FETCH_DIR WRITE_DIR OUT.txt "COMMANDS"

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
           "stabilize.hip"]
CALIBRATION_BYTES = 64 << 20  # the benchmark's plain device-to-device copy


def source_digest() -> str:
    h = hashlib.sha256()
    for name in SOURCES:
        with open(os.path.join(PKG, "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def launch_of(kernel_name: str) -> str | None:
    """'launch1'..'launch4' for the step kernels (last template argument),
    'stab_fix_v' for the stabilisation's pass over V, else None."""
    m = re.search(r"step_kernel<[^<>]*?,\s*(\d)\s*>", kernel_name)
    if m:
        return f"launch{m.group(1)}"
    return "stab_fix_v" if "stab_fix_v_kernel" in kernel_name else None


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
    sums, counts = {}, {}
    fill_seen = False
    copy_val = None
    for _, name, val in rows:
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
    rows = con.execute("select name, count(*), sum(duration), avg(duration), min(duration), "
                       "max(duration) from kernels group by name order by sum(duration) desc").fetchall()
    total = sum(r[2] for r in rows) or 1.0
    lines = ["# Kernel time summary (rocprofv3 --kernel-trace --stats)", "",
             f"Command: `{command}`", "",
             "Durations are per dispatch, kernel execution only (ns from the trace, shown in us).", "",
             "| Kernel | Launch | Calls | Total (us) | Average (us) | Min (us) | Max (us) | Share |",
             "|---|---|---|---|---|---|---|---|"]
    for name, calls, tot, avg, mn, mx in rows:
        short = name if len(name) < 90 else name[:87] + "..."
        lines.append(f"| `{short}` | {launch_of(name) or ''} | {calls} | {tot / 1e3:.1f} | "
                     f"{avg / 1e3:.2f} | {mn / 1e3:.2f} | {mx / 1e3:.2f} | {100 * tot / total:.1f}% |")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")


def main(argv):
    if len(argv) >= 4 and argv[0] == "stats":
        write_stats(argv[1], argv[2], argv[3])
    elif len(argv) >= 5 and argv[0] == "traffic":
        print(json.dumps(write_traffic(argv[1], argv[2], argv[3], argv[4])))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
