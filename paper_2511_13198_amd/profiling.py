"""Turn rocprofv3 output into the kernel profile summary of a workload.

Inputs are rocprofv3 output directories (CSV format):
  * a kernel trace with --stats (average duration per kernel);
  * a counter pass with SQ_WAVE_CYCLES, SQ_BUSY_CYCLES, SQ_WAIT_ANY,
    SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_ANY, SQ_ACTIVE_INST_VALU,
    SQ_ACTIVE_INST_LDS, SQ_VALU_MFMA_BUSY_CYCLES and GRBM_GUI_ACTIVE;
  * one FETCH_SIZE pass and one WRITE_SIZE pass of the workload, and the
    same two counters for a plain 1 GiB device copy (bench.py
    --copy-calibration-mib 1024), which give the factor between counter
    kilobytes and bytes actually moved.

Output: a markdown table (stdout or --md) and a JSON record of the HBM bytes
per launch of each library kernel, stamped with a hash of the kernel sources
so that bench.py can tell whether the counters still describe the kernels it
runs.

Usage:
  python -m paper_2511_13198_amd.profiling --trace DIR --pmc DIR --fetch DIR --write DIR \
      --copy-fetch DIR --copy-write DIR --copy-mib 1024 --workload NAME --md OUT.md --json OUT.json
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
from typing import Dict, List

_HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY_KERNELS = ("plan_kernel", "fwd_kernel", "bwd_dkdv_kernel", "bwd_dq_kernel",
                   "split_merge_kernel", "split_sum_kernel")


def code_text(src: str) -> str:
    """C++ source with comments removed and whitespace collapsed: the part of a
    kernel source that can change the compiled code.  (String literals in the
    kernel sources hold no comment markers.)"""
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def source_hash() -> str:
    """sha256 over the code (comments and layout aside) of the HIP sources the
    library is built from, sorted by name."""
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(_HERE, "csrc", "*"))):
        if p.endswith((".hip", ".hpp", ".h")):
            h.update(os.path.basename(p).encode())
            h.update(code_text(open(p).read()).encode())
    return h.hexdigest()


def short_name(kernel: str) -> str:
    """Library kernel name (e.g. 'fwd_kernel') of a demangled kernel string."""
    for k in LIBRARY_KERNELS:
        if f"pdy::{k}" in kernel:
            return k
    return ""


def _csv(d: str, suffix: str) -> List[dict]:
    paths = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not paths:
        raise FileNotFoundError(f"no *{suffix} under {d}")
    rows: List[dict] = []
    for p in paths:
        rows += list(csv.DictReader(open(p)))
    return rows


def counters(d: str) -> Dict[str, Dict[str, List[float]]]:
    """kernel -> counter -> per-dispatch values."""
    out: Dict[str, Dict[str, Dict[str, float]]] = collections.defaultdict(
        lambda: collections.defaultdict(dict))
    for r in _csv(d, "counter_collection.csv"):
        out[r["Kernel_Name"]][r["Counter_Name"]][r["Dispatch_Id"]] = float(r["Counter_Value"])
    return {k: {c: list(v.values()) for c, v in cs.items()} for k, cs in out.items()}


def clock_ghz(d: str) -> Dict[str, float]:
    """kernel -> mean shader clock (GHz) over its dispatches in a counter pass
    with GRBM_GUI_ACTIVE: the counter (summed over the 8 XCDs) / 8 / the
    dispatch's duration."""
    per: Dict[str, List[float]] = collections.defaultdict(list)
    for r in _csv(d, "counter_collection.csv"):
        if r["Counter_Name"] != "GRBM_GUI_ACTIVE" or not r.get("End_Timestamp"):
            continue
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
        if dur > 0:
            per[r["Kernel_Name"]].append(float(r["Counter_Value"]) / 8.0 / dur / 1e9)
    return {k: _mean(v) for k, v in per.items()}


def kernel_stats(d: str) -> Dict[str, dict]:
    out = {}
    for r in _csv(d, "kernel_stats.csv"):
        out[r["Name"]] = {"calls": int(r["Calls"]), "avg_ns": float(r["AverageNs"]),
                          "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"])}
    return out


def _mean(x):
    return sum(x) / len(x) if x else float("nan")


def copy_scale(d: str, counter: str, copy_mib: int) -> float:
    """Bytes per counter unit: (copy size) / (counter KiB x 1024) for the copy kernel."""
    for k, cs in counters(d).items():
        if "copyBuffer" in k and counter in cs:
            return copy_mib * 2.0 ** 20 / (_mean(cs[counter]) * 1024.0)
    raise ValueError(f"no copy kernel with {counter} in {d}")


def summarize(a) -> dict:
    stats = kernel_stats(a.trace)
    pmc = counters(a.pmc)
    clocks = clock_ghz(a.pmc)
    fetch = counters(a.fetch)
    write = counters(a.write)
    fs = copy_scale(a.copy_fetch, "FETCH_SIZE", a.copy_mib)
    ws = copy_scale(a.copy_write, "WRITE_SIZE", a.copy_mib)
    rec = {"workload": a.workload, "source_sha256": source_hash(), "fetch_scale": fs,
           "write_scale": ws, "kernels": {}}
    for full, st in stats.items():
        k = short_name(full)
        if not k:
            continue
        e = {"kernel": full, "calls": st["calls"], "avg_ms": st["avg_ns"] / 1e6}
        p = pmc.get(full, {})
        if p:
            grbm = _mean(p.get("GRBM_GUI_ACTIVE", []))  # summed over the 8 XCDs
            wave = _mean(p.get("SQ_WAVE_CYCLES", []))
            e["mfma_busy_pct"] = 100.0 * _mean(p.get("SQ_VALU_MFMA_BUSY_CYCLES", [])) / (
                grbm / 8.0 * 1024.0) if grbm else None
            e["clock_ghz"] = clocks.get(full)
            for c in ("SQ_ACTIVE_INST_ANY", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY",
                      "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS"):
                e[c.lower() + "_pct_of_wave"] = 100.0 * _mean(p.get(c, [])) / wave if wave else None
        if full in fetch:
            e["fetch_bytes"] = _mean(fetch[full]["FETCH_SIZE"]) * 1024.0 * fs
        if full in write:
            e["write_bytes"] = _mean(write[full]["WRITE_SIZE"]) * 1024.0 * ws
        rec["kernels"][k] = e
    return rec


def markdown(rec: dict, commands: List[str]) -> str:
    lines = [f"# Kernel profile: {rec['workload']}, MI355X", "",
             f"Kernel code sha256 (comments and layout aside) `{rec['source_sha256']}`.", "", "Commands:", ""]
    lines += [f"- `{c}`" for c in commands]
    lines += ["", f"Copy calibration: FETCH_SIZE x {rec['fetch_scale']:.3f}, "
              f"WRITE_SIZE x {rec['write_scale']:.3f} (bytes per counter KiB / 1024).", "",
              "| kernel | calls | avg ms | clock GHz | MFMA busy % | issuing % | waiting (waitcnt/barrier) % "
              "| waiting to issue % | VALU active % | LDS active % | HBM fetch GB | HBM write GB |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|"]

    def f(x, fmt):
        return "" if x is None else format(x, fmt)
    for k in LIBRARY_KERNELS:
        e = rec["kernels"].get(k)
        if not e:
            continue
        lines.append("| " + " | ".join([
            k, str(e["calls"]), f(e["avg_ms"], ".3f"), f(e.get("clock_ghz"), ".2f"),
            f(e.get("mfma_busy_pct"), ".1f"),
            f(e.get("sq_active_inst_any_pct_of_wave"), ".1f"),
            f(e.get("sq_wait_any_pct_of_wave"), ".1f"),
            f(e.get("sq_wait_inst_any_pct_of_wave"), ".1f"),
            f(e.get("sq_active_inst_valu_pct_of_wave"), ".1f"),
            f(e.get("sq_active_inst_lds_pct_of_wave"), ".1f"),
            f(e.get("fetch_bytes", 0) / 1e9, ".3f"), f(e.get("write_bytes", 0) / 1e9, ".3f"),
        ]) + " |")
    lines += ["", "MFMA busy % = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE per XCD x 1024 SIMDs); "
              "the other percentages are of SQ_WAVE_CYCLES (time waves are resident).  Clock = "
              "GRBM_GUI_ACTIVE per XCD / dispatch duration in the counter pass (kernels run "
              "slightly slower under counter collection); the clock-adjusted bf16 peak is "
              "2516.6 TFLOP/s x clock / 2.4 GHz.", ""]
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    for n in ("trace", "pmc", "fetch", "write", "copy-fetch", "copy-write", "workload"):
        ap.add_argument(f"--{n}", required=True)
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--md")
    ap.add_argument("--json")
    ap.add_argument("--command", action="append", default=[],
                    help="command lines to record in the summary (repeatable)")
    a = ap.parse_args(argv)
    rec = summarize(a)
    md = markdown(rec, a.command)
    if a.md:
        open(a.md, "w").write(md + "\n")
    else:
        print(md)
    if a.json:
        with open(a.json, "w") as fh:
            json.dump(rec, fh, indent=1)


if __name__ == "__main__":
    main()
