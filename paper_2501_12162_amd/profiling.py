"""Summaries of rocprofv3 output for the committed profiles.

Usage (on an MI355X, after the runs named in each summary's header):

  python -m paper_2501_12162_amd.profiling stats  <kernel_stats.csv> <out.md> "<command>" [<kernel_trace.csv> <warmup> <steps>]
  python -m paper_2501_12162_amd.profiling traffic <fetch_dir> <write_dir> <workload> <out.json> "<commands>"
  python -m paper_2501_12162_amd.profiling traffic-sampled <fetch_dir> <write_dir> <workload> <out.json> "<commands>"
  python -m paper_2501_12162_amd.profiling counters <out.json> <workload> "<commands>" <dir> [<dir> ...]

``traffic`` reads the per-dispatch FETCH_SIZE and WRITE_SIZE counters (KiB) of
the tree-attention and argmax kernels, scales each by the factor that makes
the bench's calibration copy (a device-to-device copy of exactly 256 MiB,
launched by bench.py before timing) read and write 256 MiB, and stores the
result with a hash of the kernel sources (comments excluded); ``bench.py``
reports it only while the sources still have that hash.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import re
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CALIB_BYTES = 256 << 20


_TRAFFIC_FILES = ("tree_attn.hip", "argmax.hip", "argmax_row.h", "accept_wave.h", "plan.h", "device_common.h",
                  "host_plan.h", "host_plan.cpp")


def _block(text: str, start: str, end: str) -> str:
    i = text.index(start)
    return text[i:text.index(end, i)]


def _code_only(text: str) -> str:
    """The text without its comments and with whitespace runs collapsed, so
    that edits to comments alone keep the hash (the sources hashed here hold
    no "//" or "/*" inside string literals)."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash() -> str:
    """sha256 over the sources that decide the measured kernels' traffic: the
    tree-attention and argmax kernels, their headers, the attention argument
    block, the host validation and planner, and the launch path (other entry
    points do not change it)."""
    h = hashlib.sha256()
    csrc = os.path.join(PKG, "csrc")
    for name in _TRAFFIC_FILES:
        with open(os.path.join(csrc, name)) as f:
            h.update(name.encode())
            h.update(_code_only(f.read()).encode())
    with open(os.path.join(csrc, "kernels.h")) as f:
        h.update(_code_only(_block(f.read(), "struct TreeAttnArgs", "};")).encode())
    with open(os.path.join(csrc, "adaserve.cpp")) as f:
        text = f.read()
    h.update(_code_only(_block(text, "int32_t tree_attn_verify_impl(",
                                     "int32_t adaserve_tree_accept(")).encode())
    return h.hexdigest()[:16]


def sampled_source_hash() -> str:
    """sha256 over the sources that decide the sampled-verification kernels'
    traffic: sampled.hip and the argument block and parts sizing it shares
    with the host."""
    h = hashlib.sha256()
    csrc = os.path.join(PKG, "csrc")
    for name in ("sampled.hip", "device_common.h"):
        with open(os.path.join(csrc, name)) as f:
            h.update(name.encode())
            h.update(_code_only(f.read()).encode())
    with open(os.path.join(csrc, "kernels.h")) as f:
        h.update(_code_only(_block(f.read(), "struct SampledArgs", "hipError_t launch_sampled_accept")).encode())
    return h.hexdigest()[:16]


def kernel_kind(name: str) -> str:
    if "tree_attn_combine" in name:
        return "tree_attn_combine"
    if "tree_attn_bf16" in name or "tree_attn_f32" in name:
        return "tree_attn"
    if "node_argmax" in name:
        return "node_argmax"
    if "tree_accept" in name:
        return "tree_accept"
    if "beam_scan" in name:
        return "beam_scan"
    if "beam_merge" in name:
        return "beam_merge"
    if "sampled_stats" in name:
        return "sampled_stats"
    if "sampled_accept" in name:
        return "sampled_accept"
    return "other"


def stats_markdown(csv_path: str, command: str) -> str:
    rows = list(csv.DictReader(open(csv_path)))
    out = ["# rocprofv3 kernel statistics", "", "Command:", "", "```", command, "```", "",
           "| kernel | calls | average (us) | min (us) | max (us) | share |", "|---|---|---|---|---|---|"]
    for r in rows:
        out.append("| %s | %s | %.2f | %.2f | %.2f | %.1f%% |" % (
            r["Name"][:90].replace("|", "/"), r["Calls"], float(r["AverageNs"]) / 1e3,
            float(r["MinNs"]) / 1e3, float(r["MaxNs"]) / 1e3, float(r["Percentage"])))
    return "\n".join(out) + "\n"


def timed_step_summary(trace_csv: str, warmup: int, steps: int) -> dict:
    """The verification launches of bench.py's timed loop, read from a
    rocprofv3 kernel trace: the tree-attention dispatches number warmup ..
    warmup + steps - 1 in dispatch order (one per step; the step's second
    launch, the merge/acceptance kernel, is the dispatch after each).  Returns
    the mean duration of each of the two launches over those steps and the
    mean start-to-start interval of consecutive steps (the GPU's time per
    step, gaps included)."""
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Dispatch_Id"]))
    attn = [i for i, r in enumerate(rows) if kernel_kind(r["Kernel_Name"]) == "tree_attn"]
    if len(attn) < warmup + steps:
        raise RuntimeError("trace holds %d attention dispatches, fewer than %d" % (len(attn), warmup + steps))
    idx = attn[warmup:warmup + steps]
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    start = [int(rows[i]["Start_Timestamp"]) for i in idx]
    res = {"steps": steps, "tree_attn_us": statistics.fmean(dur(rows[i]) for i in idx),
           "start_to_start_us": (start[-1] - start[0]) / 1e3 / (steps - 1)}
    nxt = [rows[i + 1] for i in idx if i + 1 < len(rows)]
    if len(nxt) == steps and all(kernel_kind(r["Kernel_Name"]) == "tree_attn_combine" for r in nxt):
        res["tree_attn_combine_us"] = statistics.fmean(dur(r) for r in nxt)
    return res


def _counter_rows(directory: str, counter: str):
    files = glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)
    rows = []
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter:
                rows.append(r)
    return rows


def _calibration_factor(rows, expect_bytes: int) -> float:
    # bench.py launches the calibration copy right before its first
    # verification step: it is the last non-library dispatch before the first
    # tree-attention dispatch.
    rows = sorted(rows, key=lambda r: int(r["Dispatch_Id"]))
    first = min(int(r["Dispatch_Id"]) for r in rows if kernel_kind(r["Kernel_Name"]) == "tree_attn")
    before = [r for r in rows if int(r["Dispatch_Id"]) < first and kernel_kind(r["Kernel_Name"]) == "other"]
    if not before:
        raise RuntimeError("calibration copy not found")
    value = float(before[-1]["Counter_Value"])
    return (expect_bytes / 1024.0) / value


def traffic_summary(fetch_dir: str, write_dir: str, workload: int, commands: str, sampled: bool = False) -> dict:
    """Calibrated HBM bytes per dispatch (medians) of the verification
    kernels, or with `sampled` of the sampled-verification kernels (their
    own source hash)."""
    fetch = _counter_rows(fetch_dir, "FETCH_SIZE")
    write = _counter_rows(write_dir, "WRITE_SIZE")
    f_factor = _calibration_factor(fetch, CALIB_BYTES)
    w_factor = _calibration_factor(write, CALIB_BYTES)
    res = {"workload": workload, "kernel_source_sha": sampled_source_hash() if sampled else kernel_source_hash(),
           "fetch_factor": f_factor, "write_factor": w_factor, "commands": commands, "kernels": {}}
    kinds = ("sampled_stats", "sampled_accept") if sampled else (
        "tree_attn", "tree_attn_combine", "node_argmax", "tree_accept")
    for kind in kinds:
        fv = [float(r["Counter_Value"]) for r in fetch if kernel_kind(r["Kernel_Name"]) == kind]
        wv = [float(r["Counter_Value"]) for r in write if kernel_kind(r["Kernel_Name"]) == kind]
        if not fv:
            continue
        fb = statistics.median(fv) * 1024 * f_factor
        wb = statistics.median(wv) * 1024 * w_factor if wv else 0.0
        res["kernels"][kind] = {"fetch_bytes": fb, "write_bytes": wb, "bytes": fb + wb,
                                "dispatches": len(fv)}
    return res


def counter_summary(dirs, workload: int, commands: str, simds: int = 1024, xcds: int = 8) -> dict:
    """Per-kernel medians over dispatches of every counter found under `dirs`
    (one rocprofv3 --pmc run each), with derived figures:

    * rocprofv3 reports each counter summed over its hardware instances, so
      GRBM_GUI_ACTIVE is the sum over the XCDs: active cycles per XCD =
      GRBM_GUI_ACTIVE / xcds, and that over the dispatch's duration is the
      clock the kernel ran at;
    * mfma_busy_frac = SQ_VALU_MFMA_BUSY_CYCLES / (cycles per XCD * SIMDs),
      the share of SIMD-cycles the matrix cores were busy;
    * mfma_bf16_flops = SQ_INSTS_VALU_MFMA_MOPS_BF16 * 512, the bf16 matrix
      work the hardware counted (padding and row-sum products included);
    * valu_per_mfma, the non-matrix vector instructions per matrix one;
    * lds_conflict_frac = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE, the share
      of LDS cycles lost to bank conflicts;
    * wait / active shares of SQ_WAVE_CYCLES (SQ_WAIT_ANY: waits on memory
      counters and barriers; SQ_WAIT_INST_ANY: waiting to issue;
      SQ_ACTIVE_INST_ANY: issuing), all in the same units."""
    per = {}
    for d in dirs:
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        for f in files:
            for r in csv.DictReader(open(f)):
                kind = kernel_kind(r["Kernel_Name"])
                if kind == "other":
                    continue
                c = per.setdefault(kind, {})
                c.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                if r.get("Start_Timestamp") and r.get("End_Timestamp"):
                    c.setdefault("duration_ns", []).append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
    res = {"workload": workload, "kernel_source_sha": kernel_source_hash(), "commands": commands,
           "kernels": {}}
    for kind, counters in per.items():
        med = {c: statistics.median(v) for c, v in counters.items()}
        k = {"counters": med, "dispatches": max(len(v) for v in counters.values())}
        gui = med.get("GRBM_GUI_ACTIVE")
        if gui:
            k["cycles_per_xcd"] = gui / xcds
            if med.get("duration_ns"):
                k["clock_ghz"] = gui / xcds / med["duration_ns"]
        if gui and "SQ_VALU_MFMA_BUSY_CYCLES" in med:
            k["mfma_busy_frac"] = med["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui / xcds * simds)
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in med:
            k["mfma_bf16_flops"] = med["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
        if "SQ_INSTS_MFMA" in med and "SQ_INSTS_VALU" in med and med["SQ_INSTS_MFMA"]:
            k["valu_per_mfma"] = (med["SQ_INSTS_VALU"] - med["SQ_INSTS_MFMA"]) / med["SQ_INSTS_MFMA"]
        if med.get("SQ_LDS_IDX_ACTIVE"):
            k["lds_conflict_frac"] = med.get("SQ_LDS_BANK_CONFLICT", 0.0) / med["SQ_LDS_IDX_ACTIVE"]
        if med.get("SQ_WAVE_CYCLES"):
            for name, key in (("SQ_WAIT_ANY", "wait_any_frac"), ("SQ_WAIT_INST_ANY", "wait_inst_frac"),
                              ("SQ_ACTIVE_INST_ANY", "active_inst_frac")):
                if name in med:
                    k[key] = med[name] / med["SQ_WAVE_CYCLES"]
        res["kernels"][kind] = k
    return res


def main(argv):
    if len(argv) >= 4 and argv[1] == "stats":
        md = stats_markdown(argv[2], argv[4] if len(argv) > 4 else "")
        if len(argv) >= 8:
            t = timed_step_summary(argv[5], int(argv[6]), int(argv[7]))
            md += ("\nTimed loop only (dispatches %d to %d of the attention kernel, from the kernel trace): "
                   "attention launch %.2f us" % (int(argv[6]), int(argv[6]) + t["steps"] - 1, t["tree_attn_us"]))
            if "tree_attn_combine_us" in t:
                md += ", second launch %.2f us" % t["tree_attn_combine_us"]
            md += ", start to start %.2f us per step.\n" % t["start_to_start_us"]
        with open(argv[3], "w") as f:
            f.write(md)
        print(md)
    elif len(argv) >= 6 and argv[1] in ("traffic", "traffic-sampled"):
        res = traffic_summary(argv[2], argv[3], int(argv[4]), argv[6] if len(argv) > 6 else "",
                              sampled=argv[1] == "traffic-sampled")
        with open(argv[5], "w") as f:
            json.dump(res, f, indent=1)
        print(json.dumps(res, indent=1))
    elif len(argv) >= 5 and argv[1] == "counters":
        # counters <out.json> <workload> "<commands>" <dir> [<dir> ...]
        res = counter_summary(argv[5:], int(argv[3]), argv[4])
        with open(argv[2], "w") as f:
            json.dump(res, f, indent=1)
        print(json.dumps(res, indent=1))
    else:
        print(__doc__)
        return 2
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv))
