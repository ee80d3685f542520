"""Summaries of rocprofv3 output for the benchmark's kernels.

Reads the CSV files of three rocprofv3 runs of bench.py (a kernel trace with
--stats, a FETCH_SIZE pass and a WRITE_SIZE pass, each with
--copy-calib-mb 1024 so that a plain elementwise kernel of known traffic is
in the same run) and writes

  profiles/<name>.md   per-kernel durations (all launches and per grid size)
                       and HBM traffic, with the commands that produced them
  profiles/traffic.json  HBM bytes per launch of the decode and prefill
                       kernels, tied to the kernel sources by a hash, read by
                       bench.py for its roofline `traffic` field

Usage:
  python -m paper_2606_11244_amd.profsum TRACE_DIR FETCH_DIR WRITE_DIR NAME \
      "TRACE_CMD" "FETCH_CMD" "WRITE_CMD"
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import json
import os
import re
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CALIB_BYTES = 1 << 30  # the calibration kernel reads and writes 1 GiB

# fp16, one token tile, any row tiles, local-EC epilogue: every launch of the
# decode pass (grouped and single calls)
DECODE_KERNEL = r"k_gemv(_group)?<0, 1, \d, 3>"
PREFILL_KERNEL = r"k_gemm<0, 1, 4>"     # fp16, EC epilogue, 256-token tiles


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in ("spear_kernels.hip", "spear_api.cpp", "spear_internal.h"):
        with open(os.path.join(ROOT, "paper_2606_11244_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _one(pattern):
    hits = glob.glob(pattern, recursive=True)
    if not hits:
        raise FileNotFoundError(pattern)
    return hits[0]


def _grid(row, gkey, wkey):
    return int(row[gkey]) // max(1, int(row[wkey]))


def counters(pmc_dir):
    """{(kernel name, workgroups): [values]} and the calibration kernel's value (KiB)."""
    rows = list(csv.DictReader(open(_one(os.path.join(pmc_dir, "**", "*counter_collection.csv")))))
    by = collections.defaultdict(list)
    calib = None
    for r in rows:
        name = r["Kernel_Name"]
        v = float(r["Counter_Value"])
        if "neg_kernel" in name:  # the calibration kernel (the run's only negation)
            calib = max(calib or 0.0, v)
        by[(name, _grid(r, "Grid_Size", "Workgroup_Size"))].append(v)
    return by, calib


def main(argv):
    trace_dir, fetch_dir, write_dir, name, tcmd, fcmd, wcmd = argv[1:8]
    stats = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_stats.csv")))))
    trace = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_trace.csv")))))
    fetch, cal_f = counters(fetch_dir)
    write, cal_w = counters(write_dir)
    if not cal_f or not cal_w:
        raise RuntimeError("calibration kernel not found in the counter runs")
    k_f = CALIB_BYTES / (cal_f * 1024.0)   # bytes per reported KiB, reads
    k_w = CALIB_BYTES / (cal_w * 1024.0)   # bytes per reported KiB, writes

    per_grid = collections.defaultdict(list)
    for r in trace:
        if "spear::" in r["Kernel_Name"]:
            key = (r["Kernel_Name"].split("(")[0].replace("void spear::", ""),
                   _grid(r, "Grid_Size_X", "Workgroup_Size_X"))
            per_grid[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)

    def traffic(kernel):
        """Mean HBM bytes per launch (reads and writes, calibrated) of a kernel."""
        tot, n = 0.0, 0
        for (nm, g), vals in fetch.items():
            if re.search(kernel, nm):
                tot += sum(vals) * 1024 * k_f
                n += len(vals)
        for (nm, g), vals in write.items():
            if re.search(kernel, nm):
                tot += sum(vals) * 1024 * k_w
        return tot / n if n else None

    lines = [f"# rocprofv3 summary: {name}", "",
             "Workload: bench.py (Llama-3.2-1B-shaped W4+EC layers, fp16, group 128, rank 16, "
             "sigmoid-linear gate): decode M=1 over 16 layers x 7 modules (q,k,v and gate,up "
             "as grouped calls), prefill M=4096 over 7 modules, W4-only reference passes; "
             "synthetic data.", "",
             "Commands (from the repository root, with TMPDIR=/tmp):", "",
             f"    {tcmd}", f"    {fcmd}", f"    {wcmd}", "",
             f"Kernel sources hash: {kernel_source_hash()}", "",
             "## Kernel durations (kernel trace, --stats)", "",
             "| kernel | calls | average us | min us | max us | share |",
             "|---|---|---|---|---|---|"]
    for r in stats[:12]:
        lines.append(f"| `{r['Name'].split('(')[0].replace('void ', '')}` | {r['Calls']} | "
                     f"{float(r['AverageNs']) / 1e3:.3f} | {float(r['MinNs']) / 1e3:.3f} | "
                     f"{float(r['MaxNs']) / 1e3:.3f} | {float(r['Percentage']):.2f}% |")
    lines += ["", "## Library kernels by grid size (workgroups): mean and median duration", "",
              "| kernel | workgroups | launches | mean us | median us |", "|---|---|---|---|---|"]
    for (k, g), v in sorted(per_grid.items()):
        v = sorted(v)
        lines.append(f"| `{k}` | {g} | {len(v)} | {sum(v) / len(v):.3f} | {v[len(v) // 2]:.3f} |")
    lines += ["", "## HBM traffic (FETCH_SIZE, WRITE_SIZE), calibrated", "",
              f"Calibration kernel (fp32 negation of 1 GiB): FETCH_SIZE {cal_f:.1f} KiB, "
              f"WRITE_SIZE {cal_w:.1f} KiB, so reads scale by {k_f:.3f} and writes by {k_w:.3f}.",
              "", "| kernel | workgroups | launches | read MB/launch | write MB/launch |",
              "|---|---|---|---|---|"]
    for (nm, g), vals in sorted(fetch.items(), key=lambda kv: kv[0][0]):
        if "spear::" not in nm:
            continue
        w = write.get((nm, g), [0.0])
        lines.append(f"| `{nm.split('(')[0].replace('void spear::', '')}` | {g} | {len(vals)} | "
                     f"{sum(vals) / len(vals) * 1024 * k_f / 1e6:.3f} | "
                     f"{sum(w) / len(w) * 1024 * k_w / 1e6:.3f} |")
    dec, pre = traffic(DECODE_KERNEL), traffic(PREFILL_KERNEL)
    lines += ["", f"Decode kernel `{DECODE_KERNEL}`: {dec / 1e6:.3f} MB per launch (mean over the "
              "decode pass's launches).",
              f"Prefill kernel `{PREFILL_KERNEL}`: {pre / 1e6:.3f} MB per launch.", ""]
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"{name}.md"), "w") as f:
        f.write("\n".join(lines))
    out = {"kernel_source_hash": kernel_source_hash(),
           "decode_kernel": DECODE_KERNEL, "decode_bytes_per_launch": round(dec),
           "prefill_kernel": PREFILL_KERNEL, "prefill_bytes_per_launch": round(pre),
           "read_scale": round(k_f, 4), "write_scale": round(k_w, 4),
           "commands": [tcmd, fcmd, wcmd]}
    with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))




# ---------------------------------------------------------------------------
# The benchmark's headline workload: the 70B-shaped model's decode (M = 1)
# and prefill (M = 4096) passes. A launch belongs to the decode pass when it
# is a GEMV (k_gemv) or an EC pre-kernel with fewer than 256 workgroups (one
# token tile), to the prefill pass when it is a GEMM (k_gemm) or an EC
# pre-kernel with 256 workgroups or more.
# ---------------------------------------------------------------------------

def _pass_of(name, grid):
    if "k_gemv" in name:
        return "decode"
    if "k_gemm" in name:
        return "prefill"
    if "k_ec<" in name:
        return "decode" if grid < 256 else "prefill"
    return None


def main70(argv):
    """profsum --llama70b TRACE_DIR FETCH_DIR WRITE_DIR SQ_DIRS NAME TRACE_CMD FETCH_CMD
    WRITE_CMD SQ_CMDS. SQ_DIRS is a comma-separated list of counter runs (or "-"),
    SQ_CMDS their commands joined by " | "."""
    trace_dir, fetch_dir, write_dir, sq_dir, name, tcmd, fcmd, wcmd, scmd = argv[2:11]
    stats = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_stats.csv")))))
    trace = list(csv.DictReader(open(_one(os.path.join(trace_dir, "**", "*kernel_trace.csv")))))
    fetch, cal_f = counters(fetch_dir)
    write, cal_w = counters(write_dir)
    if not cal_f or not cal_w:
        raise RuntimeError("calibration kernel not found in the counter runs")
    k_f = CALIB_BYTES / (cal_f * 1024.0)
    k_w = CALIB_BYTES / (cal_w * 1024.0)
    dur = collections.defaultdict(list)
    for r in trace:
        if "spear::" in r["Kernel_Name"]:
            nm = r["Kernel_Name"].split("(")[0].replace("void spear::", "")
            dur[(nm, _grid(r, "Grid_Size_X", "Workgroup_Size_X"))].append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    byp = {"decode": [0.0, 0], "prefill": [0.0, 0]}
    rows = []
    for (nm, g), vals in sorted(fetch.items(), key=lambda kv: kv[0][0]):
        if "spear::" not in nm:
            continue
        short = nm.split("(")[0].replace("void spear::", "")
        w = write.get((nm, g), [0.0])
        rd = sum(vals) / len(vals) * 1024 * k_f
        wr = sum(w) / len(w) * 1024 * k_w
        p = _pass_of(short, g)
        if p:
            byp[p][0] += (rd + wr) * len(vals)
            byp[p][1] += len(vals)
        rows.append((short, g, len(vals), rd, wr, p))
    sq = {}
    for one_dir in ([] if not sq_dir or sq_dir == "-" else sq_dir.split(",")):
        srows = list(csv.DictReader(open(_one(os.path.join(one_dir, "**", "*counter_collection.csv")))))
        for r in srows:
            nm = r["Kernel_Name"].split("(")[0].replace("void spear::", "")
            if "spear::" not in r["Kernel_Name"]:
                continue
            key = (nm, _grid(r, "Grid_Size", "Workgroup_Size"))
            sq.setdefault(key, collections.defaultdict(list))[r["Counter_Name"]].append(
                float(r["Counter_Value"]))
    lines = [f"# rocprofv3 summary: {name}", "",
             "Workload: bench.py's headline, the Llama-2-70B-shaped model resident in HBM (80 "
             "layers x q,k,v,o,gate,up,down, group-128 4-bit codes, device-random), EC rank 64 "
             "with the sigmoid-linear gate on a seeded 25% of the modules: decode pass at M = 1 "
             "and prefill pass at M = 4096, every call on its AUTO path; synthetic data.", "",
             "Commands (from the repository root, with TMPDIR=/tmp):", "",
             f"    {tcmd}", f"    {fcmd}", f"    {wcmd}"] + [f"    {c.strip()}" for c in (scmd.split(" | ") if sq else [])] + [
             "", f"Kernel sources hash: {kernel_source_hash()}", "",
             "## Kernel durations (kernel trace, --stats)", "",
             "| kernel | calls | average us | min us | max us | share |",
             "|---|---|---|---|---|---|"]
    for r in stats[:14]:
        lines.append(f"| `{r['Name'].split('(')[0].replace('void ', '')}` | {r['Calls']} | "
                     f"{float(r['AverageNs']) / 1e3:.3f} | {float(r['MinNs']) / 1e3:.3f} | "
                     f"{float(r['MaxNs']) / 1e3:.3f} | {float(r['Percentage']):.2f}% |")
    lines += ["", "## Library kernels by grid size (workgroups): launches and duration", "",
              "| kernel | workgroups | pass | launches | mean us | median us |",
              "|---|---|---|---|---|---|"]
    per_pass_t = {"decode": [0.0, 0], "prefill": [0.0, 0]}
    for (k, g), v in sorted(dur.items()):
        v = sorted(v)
        p = _pass_of(k, g)
        if p:
            per_pass_t[p][0] += sum(v)
            per_pass_t[p][1] += len(v)
        lines.append(f"| `{k}` | {g} | {p or '-'} | {len(v)} | {sum(v) / len(v):.3f} | "
                     f"{v[len(v) // 2]:.3f} |")
    lines += [""]
    for p, (t, n) in per_pass_t.items():
        if n:
            lines.append(f"Mean duration of a {p}-pass launch (kernel trace): {t / n:.3f} us "
                         f"over {n} launches.")
    lines += ["", "## HBM traffic (FETCH_SIZE, WRITE_SIZE), calibrated", "",
              f"Calibration kernel (fp32 negation of 1 GiB): FETCH_SIZE {cal_f:.1f} KiB, "
              f"WRITE_SIZE {cal_w:.1f} KiB, so reads scale by {k_f:.3f} and writes by {k_w:.3f}.",
              "", "| kernel | workgroups | pass | launches | read MB/launch | write MB/launch |",
              "|---|---|---|---|---|---|"]
    for (short, g, n, rd, wr, p) in rows:
        lines.append(f"| `{short}` | {g} | {p or '-'} | {n} | {rd / 1e6:.3f} | {wr / 1e6:.3f} |")
    dec = byp["decode"][0] / max(1, byp["decode"][1])
    pre = byp["prefill"][0] / max(1, byp["prefill"][1])
    lines += ["", f"Decode pass: {dec / 1e6:.3f} MB per launch (all its launches).",
              f"Prefill pass: {pre / 1e6:.3f} MB per launch (all its launches).", ""]
    if sq:
        names = sorted({c for v in sq.values() for c in v})
        lines += ["## SQ counters (one pass, mean per launch)", "",
                  "MFMA utilisation = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs x "
                  "256 CUs x 4 SIMDs): the share of the SIMDs' cycles, while the kernel ran, in "
                  "which the matrix unit was busy. GRBM_GUI_ACTIVE comes summed over the eight "
                  "XCDs (divided by 8 it matches the kernel's duration at 2.4 GHz) and "
                  "SQ_VALU_MFMA_BUSY_CYCLES summed over the SIMDs. MFMA flops = "
                  "SQ_INSTS_VALU_MFMA_MOPS_F16 x 512 (= SQ_INSTS_MFMA x 16384 for the 16x16x32 "
                  "MFMA).", "",
                  "| kernel | workgroups | " + " | ".join(names) + " | MFMA utilisation | "
                  "MFMA TFLOP per launch |",
                  "|---|---|" + "---|" * len(names) + "---|---|"]
        for (k, g), cs in sorted(sq.items()):
            means = {c: sum(v) / len(v) for c, v in cs.items()}
            gui = means.get("GRBM_GUI_ACTIVE", 0.0)
            util = (means.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (gui / 8 * 256 * 4)) if gui else float("nan")
            tfl = means.get("SQ_INSTS_VALU_MFMA_MOPS_F16", 0.0) * 512 / 1e12
            lines.append(f"| `{k}` | {g} | " + " | ".join(f"{means.get(c, 0):,.0f}" for c in names)
                         + f" | {util:.3f} | {tfl:.4f} |")
        lines += [""]
    os.makedirs(os.path.join(ROOT, "profiles"), exist_ok=True)
    with open(os.path.join(ROOT, "profiles", f"{name}.md"), "w") as f:
        f.write("\n".join(lines))
    out = {"kernel_source_hash": kernel_source_hash(),
           "workload": "llama-2-70b-shaped model, decode M=1 and prefill M=4096 passes",
           "decode_kernel": "every decode-pass launch (k_gemv*, k_ec with < 256 workgroups)",
           "decode_bytes_per_launch": round(dec),
           "prefill_kernel": "every prefill-pass launch (k_gemm*, k_ec with >= 256 workgroups)",
           "prefill_bytes_per_launch": round(pre),
           "read_scale": round(k_f, 4), "write_scale": round(k_w, 4),
           "commands": [tcmd, fcmd, wcmd] + ([c.strip() for c in scmd.split(" | ")] if sq else [])}
    with open(os.path.join(ROOT, "profiles", "traffic.json"), "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out))


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--llama70b":
        main70(sys.argv)
    else:
        main(sys.argv)
