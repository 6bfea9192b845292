"""Summaries of rocprofv3 result databases (kernel trace and PMC passes).

    python -m paper_1804_00344_amd.profsum trace DB --title T --cmd CMD > profiles/x.md
    python -m paper_1804_00344_amd.profsum traffic FETCH_DB WRITE_DB --preset P --calib-mib N \
        --kernel SUBSTR --cmd CMD [--json profiles/traffic.json] > profiles/y.md

`traffic` scales the per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of the selected kernel by the
ratio of known bytes to counted bytes of a plain elementwise copy of N MiB (read N, write N)
run in the same process, and records the result with a hash of the kernel's source file.
"""
from __future__ import annotations

import argparse
import collections
import hashlib
import json
import os
import re
import sqlite3
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GEMM_SRC = os.path.join(ROOT, "paper_1804_00344_amd", "csrc", "mt_gemm.hip")


def short(name: str) -> str:
    name = re.sub(r"\(.*\)$", "", name)
    return name.replace("HIP_vector_type", "vec")[:90]


def trace(db, title, cmd):
    cur = sqlite3.connect(db).cursor()
    rows = list(cur.execute("select name, total_calls, total_duration, average, percentage from top_kernels"))
    out = [f"# {title}", "", f"Command: `{cmd}`", "",
           "| kernel | calls | total us | avg us | % |", "|---|---:|---:|---:|---:|"]
    for name, calls, tot, avg, pct in rows:
        out.append(f"| `{short(name)}` | {calls} | {tot:.1f} | {avg:.2f} | {pct:.2f} |")
    return "\n".join(out) + "\n"


def _per_kernel(db):
    cur = sqlite3.connect(db).cursor()
    agg = collections.defaultdict(list)
    for name, val in cur.execute("select kernel_name, value from counters_collection"):
        agg[name].append(float(val))
    return agg


def traffic(fetch_db, write_db, preset, calib_mib, kernel, cmd, json_path=None):
    f = _per_kernel(fetch_db)
    w = _per_kernel(write_db)
    calib_bytes = calib_mib * (1 << 20)

    def calib(agg):
        # the calibration copy is the single largest elementwise dispatch
        best = max((max(v), n) for n, v in agg.items() if "elementwise" in n)
        return calib_bytes / (best[0] * 1024.0), best[1]

    ff, fname = calib(f)
    wf, wname = calib(w)
    sel_f = [v for n, vs in f.items() if kernel in n for v in vs]
    sel_w = [v for n, vs in w.items() if kernel in n for v in vs]
    if not sel_f or not sel_w:
        raise SystemExit(f"kernel {kernel!r} not found")
    kf = sum(sel_f) / len(sel_f) * 1024.0 * ff
    kw = sum(sel_w) / len(sel_w) * 1024.0 * wf
    src_hash = hashlib.sha256(open(GEMM_SRC, "rb").read()).hexdigest()[:16]
    md = [f"# HBM traffic of `{kernel}` ({preset})", "", f"Command: `{cmd}`", "",
          f"Calibration: elementwise copy of {calib_mib} MiB (`{short(fname)}`) counted "
          f"{calib_bytes / ff / 2**20:.1f} MiB fetched and {calib_bytes / wf / 2**20:.1f} MiB written; "
          f"scale factors fetch x{ff:.3f}, write x{wf:.3f}.", "",
          "| counter | dispatches | raw KiB/dispatch | calibrated MB/dispatch |", "|---|---:|---:|---:|",
          f"| FETCH_SIZE | {len(sel_f)} | {sum(sel_f) / len(sel_f):.0f} | {kf / 1e6:.2f} |",
          f"| WRITE_SIZE | {len(sel_w)} | {sum(sel_w) / len(sel_w):.0f} | {kw / 1e6:.2f} |",
          "", f"Total per launch: {(kf + kw) / 1e6:.2f} MB (source hash {src_hash})."]
    if json_path:
        data = json.load(open(json_path)) if os.path.exists(json_path) else {}
        data.setdefault(preset, {})["vocab_gemm"] = {
            "bytes_per_launch": round(kf + kw), "fetch_bytes": round(kf), "write_bytes": round(kw),
            "fetch_scale": round(ff, 4), "write_scale": round(wf, 4), "source_hash": src_hash, "command": cmd}
        json.dump(data, open(json_path, "w"), indent=1, sort_keys=True)
    return "\n".join(md) + "\n"


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd_name", required=True)
    t = sub.add_parser("trace")
    t.add_argument("db")
    t.add_argument("--title", default="Kernel trace")
    t.add_argument("--cmd", default="")
    r = sub.add_parser("traffic")
    r.add_argument("fetch_db")
    r.add_argument("write_db")
    r.add_argument("--preset", required=True)
    r.add_argument("--calib-mib", type=int, required=True)
    r.add_argument("--kernel", required=True)
    r.add_argument("--cmd", default="")
    r.add_argument("--json")
    a = ap.parse_args()
    if a.cmd_name == "trace":
        sys.stdout.write(trace(a.db, a.title, a.cmd))
    else:
        sys.stdout.write(traffic(a.fetch_db, a.write_db, a.preset, a.calib_mib, a.kernel, a.cmd, a.json))


if __name__ == "__main__":
    main()
