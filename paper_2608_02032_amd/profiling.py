"""Summaries of rocprofv3 output for the committed profiles/ directory.

    python -m paper_2608_02032_amd.profiling trace  <kernel_stats.csv> <out.md> "<command>"
    python -m paper_2608_02032_amd.profiling traffic <fetch counter_collection.csv>
           <write counter_collection.csv> <copy bytes> <out.json> <out.md> "<commands>"

    python -m paper_2608_02032_amd.profiling mfma <counter_collection.csv> <kernel_stats.csv>
           <out.json> <out.md> "<command>"

`traffic` turns FETCH_SIZE / WRITE_SIZE (KiB per dispatch) into bytes per
launch of each library kernel.  Each counter is scaled by what it reads for a
plain device copy of known size run in the same process (the copy kernel moves
`copy bytes` in and out), so counter units and partial coverage cancel.  The
JSON records a hash of every kernel source file, and bench.py reports the
traffic of a kernel only while those sources are unchanged.
"""
from __future__ import annotations

import csv
import hashlib
import json
import os
import re
import sys
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "hbm_traffic.json")
MFMA_JSON = os.path.join(ROOT, "profiles", "mfma_counters.json")
# MI355X: GRBM_GUI_ACTIVE comes back summed over the 8 XCDs; 1024 SIMDs
# (256 CUs x 4) each report SQ_VALU_MFMA_BUSY_CYCLES.
N_XCD = 8
N_SIMD = 1024
PEAK_BF16_TFLOPS = 2500.0


def source_hash() -> str:
    h = hashlib.sha256()
    for name in sorted(os.listdir(CSRC)):
        if name.endswith((".hip", ".hpp", ".cpp")):
            with open(os.path.join(CSRC, name), "rb") as fh:
                h.update(name.encode())
                h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_short(name: str):
    """Short kernel name (k_...) from a mangled or demangled library symbol."""
    if "dart" not in name:
        return None
    # mangled: a length-prefixed identifier after the namespaces
    m = re.search(r"(\d+)(k_[A-Za-z0-9_]+)", re.sub(r"\d+_GLOBAL__N_1", "", name))
    if m and int(m.group(1)) <= len(m.group(2)):
        return m.group(2)[:int(m.group(1))]
    m = re.search(r"(k_[A-Za-z0-9_]+)", name)
    return m.group(1) if m else None


def trace_summary(stats_csv: str, out_md: str, command: str) -> str:
    rows = list(csv.DictReader(open(stats_csv)))
    lines = ["# Kernel trace", "", "Command:", "", "```", command, "```", "",
             "Library kernels only.", "", "| kernel | calls | avg us | min us | max us |",
             "|---|---|---|---|---|"]
    for r in rows:
        k = kernel_short(r["Name"])
        if not k:
            continue
        lines.append("| %s | %s | %.1f | %.1f | %.1f |" % (
            k, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3))
    text = "\n".join(lines) + "\n"
    with open(out_md, "w") as fh:
        fh.write(text)
    return text


def _per_kernel(csv_path: str, counter: str):
    vals = defaultdict(list)
    copy_vals = []
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter:
            continue
        v = float(r["Counter_Value"])
        if "copyBuffer" in r["Kernel_Name"]:
            copy_vals.append(v)
        k = kernel_short(r["Kernel_Name"])
        if k:
            vals[k].append(v)
    return vals, copy_vals


def traffic_summary(fetch_csv: str, write_csv: str, copy_bytes: int, out_json: str, out_md: str,
                    commands: str) -> dict:
    fetch, fcopy = _per_kernel(fetch_csv, "FETCH_SIZE")
    write, wcopy = _per_kernel(write_csv, "WRITE_SIZE")
    # the calibration copy is the largest copyBuffer dispatch
    f_ref = max(fcopy) * 1024.0
    w_ref = max(wcopy) * 1024.0
    f_scale = copy_bytes / f_ref
    w_scale = copy_bytes / w_ref
    out = {"source_hash": source_hash(), "copy_bytes": copy_bytes,
           "fetch_scale": f_scale, "write_scale": w_scale, "kernels": {}}
    lines = ["# HBM traffic per launch (rocprofv3 FETCH_SIZE / WRITE_SIZE)", "",
             "Commands:", "", "```", commands, "```", "",
             "Scale factors from a plain %d-byte device copy in the same process: FETCH_SIZE x %.3f, "
             "WRITE_SIZE x %.3f." % (copy_bytes, f_scale, w_scale), "",
             "| kernel | dispatches | fetch MB | write MB |", "|---|---|---|---|"]
    for k in sorted(set(fetch) | set(write)):
        fv = sum(fetch.get(k, [0.0])) / max(len(fetch.get(k, [])), 1) * 1024.0 * f_scale
        wv = sum(write.get(k, [0.0])) / max(len(write.get(k, [])), 1) * 1024.0 * w_scale
        out["kernels"][k] = {"fetch_bytes": fv, "write_bytes": wv, "traffic_bytes": fv + wv}
        lines.append("| %s | %d | %.1f | %.1f |" % (k, len(fetch.get(k, [])), fv / 1e6, wv / 1e6))
    with open(out_json, "w") as fh:
        json.dump(out, fh, indent=1)
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    return out


def traffic_for(kernel: str):
    """Measured HBM bytes per launch of `kernel`, or None when no counters were
    taken for the current kernel sources."""
    if not os.path.exists(TRAFFIC_JSON):
        return None
    d = json.load(open(TRAFFIC_JSON))
    if d.get("source_hash") != source_hash():
        return None
    k = d["kernels"].get(kernel)
    return None if k is None else k["traffic_bytes"]


def mfma_summary(pmc_csv: str, stats_csv: str, out_json: str, out_md: str, command: str) -> dict:
    """Per kernel: MFMA-busy fraction of every SIMD's cycles while the kernel
    ran (SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 x 1024)), the bf16
    MFMA flops it executed (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512), the shader
    clock (GRBM_GUI_ACTIVE / 8 over the traced duration) and the executed
    TFLOP/s."""
    vals = defaultdict(lambda: defaultdict(list))
    for r in csv.DictReader(open(pmc_csv)):
        k = kernel_short(r["Kernel_Name"])
        if k:
            vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    dur = {}
    for r in csv.DictReader(open(stats_csv)):
        k = kernel_short(r["Name"])
        if k:
            dur[k] = float(r["AverageNs"]) * 1e-9
    mean = lambda v: sum(v) / len(v) if v else 0.0
    out = {"source_hash": source_hash(), "kernels": {}}
    lines = ["# MFMA counters per launch (rocprofv3 --pmc)", "", "Commands:", "", "```", command, "```",
             "", "busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / %d x %d SIMDs); "
             "executed = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 flops per launch; clock = GRBM_GUI_ACTIVE / %d "
             "over the kernel-trace average duration." % (N_XCD, N_SIMD, N_XCD), "",
             "| kernel | launches | avg us | MFMA busy | bf16 GFLOP executed | executed TFLOP/s | clock GHz |",
             "|---|---|---|---|---|---|---|"]
    for k in sorted(vals):
        c = vals[k]
        gui = mean(c.get("GRBM_GUI_ACTIVE", [])) / N_XCD
        busy = mean(c.get("SQ_VALU_MFMA_BUSY_CYCLES", []))
        mops = mean(c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", []))
        frac = busy / (gui * N_SIMD) if gui > 0 else None
        flops = mops * 512.0
        d = dur.get(k)
        tf = flops / d / 1e12 if d else None
        ghz = gui / d / 1e9 if d else None
        out["kernels"][k] = {"mfma_busy": frac, "bf16_flops": flops, "avg_s": d,
                             "executed_tflops": tf, "clock_ghz": ghz}
        lines.append("| %s | %d | %s | %s | %.1f | %s | %s |" % (
            k, len(c.get("SQ_VALU_MFMA_BUSY_CYCLES", [])), "%.1f" % (d * 1e6) if d else "-",
            "%.1f %%" % (100 * frac) if frac is not None else "-", flops / 1e9,
            "%.0f" % tf if tf else "-", "%.2f" % ghz if ghz else "-"))
    with open(out_json, "w") as fh:
        json.dump(out, fh, indent=1)
    with open(out_md, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    return out


def mfma_for(kernel: str):
    """Counter-measured MFMA-busy fraction of `kernel`, or None when no
    counters were taken for the current kernel sources."""
    if not os.path.exists(MFMA_JSON):
        return None
    d = json.load(open(MFMA_JSON))
    if d.get("source_hash") != source_hash():
        return None
    k = d["kernels"].get(kernel)
    return None if k is None or k["mfma_busy"] is None else round(k["mfma_busy"], 4)


def instmix_summary(pass1_csv: str, pass2_csv: str, out_md: str, commands: str) -> str:
    """Per kernel and wave: instructions issued by class (SQ_INSTS_VALU,
    SQ_INSTS_MFMA, SQ_INSTS_SALU, SQ_INSTS_LDS), the share
    of wave lifetime spent in s_waitcnt (SQ_WAIT_ANY) and waiting to issue
    (SQ_WAIT_INST_ANY), the share of LDS-active cycles lost to bank conflicts,
    and the mean wave lifetime (SQ_WAVE_CYCLES counts every 4 cycles)."""
    vals = defaultdict(lambda: defaultdict(list))
    for path in (pass1_csv, pass2_csv):
        for r in csv.DictReader(open(path)):
            k = kernel_short(r["Kernel_Name"])
            if k:
                vals[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    mean = lambda v: sum(v) / len(v) if v else float("nan")
    lines = ["# Instruction mix and stalls per wave (rocprofv3 --pmc, SQ counters)", "", "Commands:", "",
             "```", commands, "```", "",
             "Per wave: issued instructions by class (SQ_INSTS_VALU, _MFMA, _SALU, _LDS); wait = s_waitcnt share of "
             "the wave lifetime (SQ_WAIT_ANY / SQ_WAVE_CYCLES), issue-wait = waiting to issue "
             "(SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES); bank = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE; "
             "lifetime = 4 SQ_WAVE_CYCLES / SQ_WAVES.", "",
             "| kernel | waves | VALU | MFMA | SALU | LDS | wait | issue-wait | LDS bank | lifetime (cycles) |",
             "|---|---|---|---|---|---|---|---|---|---|"]
    for k in sorted(vals):
        c = {n: mean(v) for n, v in vals[k].items()}
        w = c.get("SQ_WAVES", float("nan"))
        wc = c.get("SQ_WAVE_CYCLES", float("nan"))
        per = lambda n: c.get(n, float("nan")) / w
        lines.append("| %s | %d | %.0f | %.0f | %.0f | %.0f | %.1f %% | %.1f %% | %.1f %% | %.0f |" % (
            k, w, per("SQ_INSTS_VALU"), per("SQ_INSTS_MFMA"), per("SQ_INSTS_SALU"), per("SQ_INSTS_LDS"),
            100 * c.get("SQ_WAIT_ANY", float("nan")) / wc, 100 * c.get("SQ_WAIT_INST_ANY", float("nan")) / wc,
            100 * c.get("SQ_LDS_BANK_CONFLICT", float("nan")) / max(c.get("SQ_LDS_IDX_ACTIVE", 1.0), 1.0),
            4 * wc / w))
    text = "\n".join(lines) + "\n"
    with open(out_md, "w") as fh:
        fh.write(text)
    return text


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        print(trace_summary(sys.argv[2], sys.argv[3], sys.argv[4]))
    elif sys.argv[1] == "traffic":
        print(json.dumps(traffic_summary(sys.argv[2], sys.argv[3], int(sys.argv[4]), sys.argv[5],
                                         sys.argv[6], sys.argv[7]), indent=1))
    elif sys.argv[1] == "instmix":
        print(instmix_summary(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5]))
    elif sys.argv[1] == "mfma":
        print(json.dumps(mfma_summary(sys.argv[2], sys.argv[3], sys.argv[4], sys.argv[5],
                                      sys.argv[6]), indent=1))
    else:
        raise SystemExit(__doc__)
