"""Summaries of rocprofv3 output for the library's kernels.

  python -m paper_2508_02751_amd.profiling stats DIR [--title T] [--cmd C]
      per-kernel call count and average / min / max duration from a
      `rocprofv3 --kernel-trace --stats --output-format csv` run, one row
      per kernel and launch grid (workgroups), from the per-dispatch trace:
      a run that launches one kernel over different grids (the whole-stack
      step and its per-layer variant) keeps them apart.

  python -m paper_2508_02751_amd.profiling traffic FETCH_DIR WRITE_DIR --copy-mib N --workload W
      HBM bytes per dispatch of each library kernel from two `--pmc` runs
      (FETCH_SIZE, WRITE_SIZE, KiB per dispatch) of workload W.  Each counter
      is scaled by what it reads for a plain device copy of N MiB in the same
      run (the largest copy dispatch), so the result is in true bytes.  Prints
      JSON keyed by kernel, with the hash of each kernel's source file so that
      a reader can tell when the kernel changed after the counters were
      taken.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")

# kernel-name fragment -> source file
KERNEL_SOURCES = {
    "small_attn_mfma": "small_attn.hip",
    "small_attn_valu": "small_attn.hip",
    "small_attn_merge": "small_attn.hip",
    "partition_kernel": "partition.hip",
    "hybrid_kernel": "hybrid.hip",
    "hybrid_group_kernel": "hybrid_group.hip",
    "hybrid_group_merge": "hybrid_group.hip",
    "match_logits": "match.hip",
    "match_rowsum": "match.hip",
    "match_scores": "match.hip",
    "match_map": "match.hip",
    "group_zq": "group_select.hip",
    "group_scores": "group_select.hip",
    "group_weights": "group_select.hip",
    "group_init": "group_select.hip",
    "accum_scores": "group_select.hip",
    "store_index": "store.hip",
    "store_copy": "store.hip",
}


def source_hash(name: str) -> str:
    return hashlib.sha256(open(os.path.join(CSRC, name), "rb").read()).hexdigest()[:16]


def short_name(full: str) -> str:
    for frag in KERNEL_SOURCES:
        if frag in full:
            i = full.index(frag)
            j = full.find("(", i)
            return full[i:j] if j > 0 else full[i:]
    return full[:60]


def _one(pattern: str) -> str:
    files = sorted(glob.glob(pattern, recursive=True))
    if not files:
        raise SystemExit(f"no file matches {pattern}")
    return files[-1]


def stats(d: str, title: str, cmd: str) -> str:
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*kernel_trace.csv")))))
    per = collections.defaultdict(list)
    total = 0.0
    for r in rows:
        ns = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
        total += ns
        if "smallkv" not in r["Kernel_Name"]:
            continue
        wgs = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]))
        per[(short_name(r["Kernel_Name"]), wgs)].append(ns)
    out = [f"# {title}", "", f"command: `{cmd}`", "",
           "| kernel | workgroups | calls | avg us | min us | max us | share of GPU time |",
           "|---|---|---|---|---|---|---|"]
    for (k, wgs), v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| {k} | {wgs} | {len(v)} | {sum(v) / len(v) / 1e3:.1f} | "
                   f"{min(v) / 1e3:.1f} | {max(v) / 1e3:.1f} | "
                   f"{100 * sum(v) / max(total, 1.0):.1f}% |")
    return "\n".join(out) + "\n"


def _fragment(full: str):
    for frag in KERNEL_SOURCES:
        if frag in full:
            return frag
    return None


def _counter(d: str, name: str):
    """Counter values per dispatch, grouped by kernel (all template instances
    of one kernel together), and the largest value a device copy read."""
    rows = list(csv.DictReader(open(_one(os.path.join(d, "**", "*counter_collection.csv")))))
    per = collections.defaultdict(list)
    copy = 0.0
    for r in rows:
        if r["Counter_Name"] != name:
            continue
        v = float(r["Counter_Value"])
        if "copyBuffer" in r["Kernel_Name"]:
            copy = max(copy, v)
        elif "smallkv" in r["Kernel_Name"]:
            frag = _fragment(r["Kernel_Name"])
            if frag:
                per[frag].append(v)
    return per, copy


def traffic(fetch_dir: str, write_dir: str, copy_mib: int) -> dict:
    fetch, copy_f = _counter(fetch_dir, "FETCH_SIZE")
    write, copy_w = _counter(write_dir, "WRITE_SIZE")
    true_kib = copy_mib * 1024.0
    ff = true_kib / copy_f if copy_f else None
    fw = true_kib / copy_w if copy_w else None
    out = {"calibration": {"copy_mib": copy_mib, "fetch_kib_read_for_copy": copy_f,
                           "write_kib_read_for_copy": copy_w, "fetch_factor": ff,
                           "write_factor": fw},
           "kernels": {}}
    for k in sorted(set(fetch) | set(write)):
        src = KERNEL_SOURCES[k]
        fk = sum(fetch.get(k, [0])) / max(1, len(fetch.get(k, [])))
        wk = sum(write.get(k, [0])) / max(1, len(write.get(k, [])))
        rb = fk * 1024 * (ff or 1.0)
        wb = wk * 1024 * (fw or 1.0)
        out["kernels"][k] = {"source": src, "dispatches": len(fetch.get(k, [])),
                             "fetch_kib": fk, "write_kib": wk, "read_bytes": rb,
                             "write_bytes": wb, "hbm_bytes_per_launch": rb + wb,
                             "source_sha256_16": source_hash(src)}
    return out


def main(argv=None):
    p = argparse.ArgumentParser()
    sub = p.add_subparsers(dest="action", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--title", default="rocprofv3 kernel statistics")
    s.add_argument("--cmd", default="")
    t = sub.add_parser("traffic")
    t.add_argument("fetch_dir")
    t.add_argument("write_dir")
    t.add_argument("--copy-mib", type=int, required=True)
    t.add_argument("--cmd", default="")
    t.add_argument("--workload", required=True, help="name of the workload the runs measured")
    a = p.parse_args(argv)
    if a.action == "stats":
        sys.stdout.write(stats(a.dir, a.title, a.cmd))
    else:
        res = traffic(a.fetch_dir, a.write_dir, a.copy_mib)
        res["workload"] = a.workload
        res["command"] = a.cmd
        json.dump(res, sys.stdout, indent=1)
        sys.stdout.write("\n")


if __name__ == "__main__":
    main()
