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


def trace(d, steps, title, cmd, note=""):
    rows = list(csv.DictReader(open(_one(d, "*kernel_stats.csv"))))
    out = [f"# {title}", "", f"Command: `{cmd}`", "",
           f"Per-step column: total duration / {steps} launches of the step (bench warmup + timed + breakdown)."
           + (f"  {note}" if note else ""), "",
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


# kernel name substring -> (class, source file): the counters of a class are valid while its
# source file hashes as recorded
KERNEL_CLASSES = [
    ("vocab_joint_threshold_kernel", "vocab_joint_threshold", "mt_vocab_joint.hip"),
    ("vocab_joint_kernel", "vocab_joint", "mt_vocab_joint.hip"),
    ("ensemble_const_kernel", "ensemble_const", "mt_ensemble.hip"),
    ("beam_finish_kernel", "beam_finish", "mt_beam.hip"),
    ("beam_nbest_kernel", "beam_nbest", "mt_beam.hip"),
    ("vocab_threshold_kernel", "vocab_threshold", "mt_vocab.hip"),
    ("vocab_kernel", "vocab_gemm", "mt_vocab.hip"),
    ("attention_order_kernel", "attention_order", "mt_attention.hip"),
    ("attention_kernel", "attention", "mt_attention.hip"),
    ("gru_cell_kernel", "gru_cell", "mt_rnn.hip"),
    ("readout_kernel", "readout", "mt_rnn.hip"),
    ("lse_kernel", "lse", "mt_rnn.hip"),
    ("row_select_kernel", "topk_row_select", "mt_topk.hip"),
    ("topk_scan_logp_kernel", "topk_scan_logp", "mt_topk.hip"),
    ("gemm_wd_kernel", "gemm_bf16", "mt_gemm.hip"),
    ("gemm_f32_kernel", "gemm_f32", "mt_gemm.hip"),
]


def _classify(name):
    for sub, cls, src in KERNEL_CLASSES:
        if sub in name:
            return cls, src
    return None, None


def _by_dispatch_shape(d, counters):
    """{(kernel name, grid size): {counter: [values per dispatch]}} of one pass."""
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(_one(d, "*counter_collection.csv"))):
        if r["Counter_Name"] in counters:
            agg[(r["Kernel_Name"], int(r["Grid_Size"]))][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return agg


def counters(fetch_dir, write_dir, mfma_dir, preset, calib_mib, cmd, json_path=None, num_simd=1024, xcds=8):
    """HBM traffic (calibrated FETCH_SIZE / WRITE_SIZE, KiB per dispatch) and matrix-core busy
    fraction (SQ_VALU_MFMA_BUSY_CYCLES over the kernel's cycles times the SIMDs; the kernel's
    cycles are GRBM_GUI_ACTIVE / number of XCDs, which count it once each) of every kernel of
    the decoder step, per (kernel, grid) shape."""
    f = _by_dispatch_shape(fetch_dir, {"FETCH_SIZE"})
    w = _by_dispatch_shape(write_dir, {"WRITE_SIZE"})
    mf = _by_dispatch_shape(mfma_dir, {"SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"}) if mfma_dir else {}
    calib_bytes = calib_mib * (1 << 20)

    def calib(agg, c):
        best = max((max(v[c]), n) for n, v in agg.items() if "elementwise" in n[0] and c in v)
        return calib_bytes / (best[0] * 1024.0), best[1][0]

    ff, fname = calib(f, "FETCH_SIZE")
    wf, wname = calib(w, "WRITE_SIZE")
    root_src = os.path.join(ROOT, "paper_1804_00344_amd", "csrc")
    rows = []
    for key in sorted(set(f) | set(w), key=lambda k: (k[0], k[1])):
        cls, src = _classify(key[0])
        if cls is None:
            continue
        fv = f.get(key, {}).get("FETCH_SIZE", [])
        wv = w.get(key, {}).get("WRITE_SIZE", [])
        if not fv or not wv:
            continue
        fb = sum(fv) / len(fv) * 1024.0 * ff
        wb = sum(wv) / len(wv) * 1024.0 * wf
        busy = None
        m = mf.get(key)
        if m and m.get("SQ_VALU_MFMA_BUSY_CYCLES") and m.get("GRBM_GUI_ACTIVE"):
            b = sum(m["SQ_VALU_MFMA_BUSY_CYCLES"]) / len(m["SQ_VALU_MFMA_BUSY_CYCLES"])
            g = sum(m["GRBM_GUI_ACTIVE"]) / len(m["GRBM_GUI_ACTIVE"])
            busy = b / (g / xcds * num_simd) if g > 0 else None
        rows.append(dict(cls=cls, src=src, name=short(key[0]), grid=key[1], n=len(fv), fetch=fb, write=wb, busy=busy,
                         src_hash=source_hash(os.path.join(root_src, src))))
    md = [f"# HBM traffic and matrix-core busy fraction per kernel ({preset})", "",
          f"Command: `{cmd}`", "",
          f"Calibration: elementwise kernel over {calib_mib} MiB (`{short(fname)}`, reads and writes {calib_mib} MiB) "
          f"counted {calib_bytes / ff / 2**20:.1f} MiB fetched and {calib_bytes / wf / 2**20:.1f} MiB written: fetch "
          f"counts are scaled by {ff:.3f}, write counts by {wf:.3f}.  MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / "
          f"(GRBM_GUI_ACTIVE / {xcds} XCDs x {num_simd} SIMDs).", "",
          "FETCH_SIZE and WRITE_SIZE count the L2's traffic to the memory fabric.  Data that the 256 MB "
          "Infinity Cache still holds from the previous step (the attention keys and context, the step's "
          "own intermediates) can be served without being counted, so small working sets may count below "
          "their algorithmic bytes; counts above them mean the kernel re-reads.",
          "",
          "| kernel | grid | dispatches | fetched MB | written MB | HBM MB per dispatch | MFMA busy |",
          "|---|---:|---:|---:|---:|---:|---:|"]
    for r in rows:
        md.append(f"| `{r['name']}` | {r['grid']} | {r['n']} | {r['fetch'] / 1e6:.2f} | {r['write'] / 1e6:.2f} | "
                  f"{(r['fetch'] + r['write']) / 1e6:.2f} | {'' if r['busy'] is None else format(r['busy'], '.3f')} |")
    md += ["", "Source hashes: " + ", ".join(sorted({f"{r['src']} {r['src_hash']}" for r in rows})) + "."]
    if json_path:
        data = json.load(open(json_path)) if os.path.exists(json_path) else {}
        ent = data.setdefault(preset, {})
        for r in rows:
            k = f"{r['cls']}@{r['grid']}"
            ent[k] = {"kernel": r["name"], "grid": r["grid"], "bytes_per_launch": round(r["fetch"] + r["write"]),
                      "fetch_bytes": round(r["fetch"]), "write_bytes": round(r["write"]),
                      "mfma_busy": None if r["busy"] is None else round(r["busy"], 4),
                      "fetch_scale": round(ff, 4), "write_scale": round(wf, 4), "source": r["src"],
                      "source_hash": r["src_hash"], "command": cmd}
            if r["cls"] in ("vocab_gemm", "vocab_joint"):
                ent[r["cls"]] = dict(ent[k])
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
    t.add_argument("--note", default="")
    r = sub.add_parser("traffic")
    r.add_argument("fetch_dir")
    r.add_argument("write_dir")
    r.add_argument("--preset", required=True)
    r.add_argument("--calib-mib", type=int, required=True)
    r.add_argument("--kernel", required=True)
    r.add_argument("--cmd", default="")
    r.add_argument("--json")
    c = sub.add_parser("counters")
    c.add_argument("fetch_dir")
    c.add_argument("write_dir")
    c.add_argument("--mfma-dir")
    c.add_argument("--preset", required=True)
    c.add_argument("--calib-mib", type=int, required=True)
    c.add_argument("--cmd", default="")
    c.add_argument("--json")
    a = ap.parse_args()
    if a.cmd_name == "counters":
        sys.stdout.write(counters(a.fetch_dir, a.write_dir, a.mfma_dir, a.preset, a.calib_mib, a.cmd, a.json))
        return
    if a.cmd_name == "trace":
        sys.stdout.write(trace(a.dir, a.steps, a.title, a.cmd, a.note))
    else:
        sys.stdout.write(traffic(a.fetch_dir, a.write_dir, a.preset, a.calib_mib, a.kernel, a.cmd, a.json))


if __name__ == "__main__":
    main()
