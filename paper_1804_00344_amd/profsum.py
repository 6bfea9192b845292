"""Summaries of rocprofv3 CSV output (kernel-trace statistics and PMC passes).

    python -m paper_1804_00344_amd.profsum trace DIR --steps N --title T --cmd CMD > profiles/x.md
    python -m paper_1804_00344_amd.profsum traffic FETCH_DIR WRITE_DIR --preset P --calib-mib N \
        --kernel SUBSTR --cmd CMD [--json profiles/traffic.json] > profiles/y.md

DIR is a rocprofv3 output directory written with `-f csv` (it holds *_kernel_stats.csv or
*_counter_collection.csv).  `traffic` scales the per-dispatch FETCH_SIZE / WRITE_SIZE (KiB)
of the selected kernel by the ratio of known bytes to counted bytes of a plain elementwise
kernel of N MiB (reads N, writes N) run in the same process, and records the result with a
hash of the vocabulary kernel's source file.
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
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
VOCAB_SRC = os.path.join(ROOT, "paper_1804_00344_amd", "csrc", "mt_vocab.hip")


def source_hash(path: str = VOCAB_SRC) -> str:
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def short(name: str) -> str:
    name = re.sub(r"\(.*\)$", "", name)
    return name.replace("HIP_vector_type", "vec")[:90]


def _one(d: str, pattern: str) -> str:
    hits = glob.glob(os.path.join(d, "**", pattern), recursive=True)
    if not hits:
        raise SystemExit(f"no {pattern} under {d}")
    return hits[0]


def trace(d, steps, title, cmd):
    rows = list(csv.DictReader(open(_one(d, "*kernel_stats.csv"))))
    out = [f"# {title}", "", f"Command: `{cmd}`", "",
           f"Per-step column: total duration / {steps} launches of the step (bench warmup + timed + breakdown).", "",
           "| kernel | calls | avg us | per step us | % |", "|---|---:|---:|---:|---:|"]
    tot = 0.0
    for r in rows:
        per = float(r["TotalDurationNs"]) / 1e3 / steps
        tot += per
        out.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {per:.2f} | "
                   f"{float(r['Percentage']):.2f} |")
    out += ["", f"Sum of kernel time per step: {tot:.1f} us."]
    return "\n".join(out) + "\n"


def _per_kernel(d):
    agg = collections.defaultdict(list)
    for r in csv.DictReader(open(_one(d, "*counter_collection.csv"))):
        agg[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return agg


def traffic(fetch_dir, write_dir, preset, calib_mib, kernel, cmd, json_path=None):
    f = _per_kernel(fetch_dir)
    w = _per_kernel(write_dir)
    calib_bytes = calib_mib * (1 << 20)

    def calib(agg):
        # the calibration kernel is the single largest elementwise dispatch
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
    src_hash = source_hash()
    md = [f"# HBM traffic of `{kernel}` ({preset})", "", f"Command: `{cmd}`", "",
          f"Calibration: elementwise kernel over {calib_mib} MiB (`{short(fname)}`, reads {calib_mib} MiB and "
          f"writes {calib_mib} MiB) counted {calib_bytes / ff / 2**20:.1f} MiB fetched and "
          f"{calib_bytes / wf / 2**20:.1f} MiB written; scale factors fetch x{ff:.3f}, write x{wf:.3f}.", "",
          "| counter | dispatches | raw KiB/dispatch | calibrated MB/dispatch |", "|---|---:|---:|---:|",
          f"| FETCH_SIZE | {len(sel_f)} | {sum(sel_f) / len(sel_f):.0f} | {kf / 1e6:.2f} |",
          f"| WRITE_SIZE | {len(sel_w)} | {sum(sel_w) / len(sel_w):.0f} | {kw / 1e6:.2f} |",
          "", f"Total per launch: {(kf + kw) / 1e6:.2f} MB (source hash {src_hash} of mt_vocab.hip)."]
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
    t.add_argument("dir")
    t.add_argument("--steps", type=float, required=True)
    t.add_argument("--title", default="Kernel trace")
    t.add_argument("--cmd", default="")
    r = sub.add_parser("traffic")
    r.add_argument("fetch_dir")
    r.add_argument("write_dir")
    r.add_argument("--preset", required=True)
    r.add_argument("--calib-mib", type=int, required=True)
    r.add_argument("--kernel", required=True)
    r.add_argument("--cmd", default="")
    r.add_argument("--json")
    a = ap.parse_args()
    if a.cmd_name == "trace":
        sys.stdout.write(trace(a.dir, a.steps, a.title, a.cmd))
    else:
        sys.stdout.write(traffic(a.fetch_dir, a.write_dir, a.preset, a.calib_mib, a.kernel, a.cmd, a.json))


if __name__ == "__main__":
    main()
