"""Summaries of rocprofv3 output for the profiles/ folder.

  python -m paper_2606_27550_amd.rocprof_summary stats <kernel_stats.csv> <out.md> "<command>"
  python -m paper_2606_27550_amd.rocprof_summary traffic <fetch.csv> <write.csv> \
      <copy_fetch.csv> <copy_write.csv> <copy_bytes> <out.md> <out.json> "<commands>"

``stats`` turns a --kernel-trace --stats CSV into a markdown table.
``counters`` averages a --pmc counter collection per kernel (name filter
optional):

  python -m paper_2606_27550_amd.rocprof_summary counters <counter_collection.csv> <out.md> "<command>" [filter]

``apiwindow`` counts the HIP and HSA API calls of a --hip-trace --hsa-trace run
inside the benchmark's timed region (between its last two hipMemGetInfo
calls) and lists every code-object load or compile call of the whole run:

  python -m paper_2606_27550_amd.rocprof_summary apiwindow <hip_api_trace.csv> <hsa_api_trace.csv> <out.md> "<command>"

``traffic`` turns FETCH_SIZE / WRITE_SIZE counter collections (KiB per
dispatch) into HBM bytes per launch, scaled by what the same counters read for
a plain device copy of known size, and records them together with the hash of
the LM-head kernel source so that a later change to the kernel invalidates them.
"""
from __future__ import annotations

import collections
import csv
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
LM_HEAD_SRCS = [os.path.join(PKG, "csrc", f) for f in
                ("lm_head.hip", "lm_head_gemm.hip", "stats.hpp", "stream_pipe.hpp")]


def lm_head_source_hash() -> str:
    """sha256 over the LM-head kernel sources (the streaming, tiled and
    device-sized kernels and their shared helpers)."""
    h = hashlib.sha256()
    for path in LM_HEAD_SRCS:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def short(name: str) -> str:
    name = name.replace("entmtp::(anonymous namespace)::", "")
    cut = name.find("(")
    return name[:cut] if cut > 0 else name


def stats(csv_path: str, out_md: str, command: str) -> None:
    rows = list(csv.DictReader(open(csv_path)))
    lines = [f"# Kernel time: `{command}`", "",
             "rocprofv3 --kernel-trace --stats summary (per-dispatch durations).", "",
             "| kernel | calls | avg us | min us | max us | % of GPU time |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        lines.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.2f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


def _counters(csv_paths):
    acc = collections.defaultdict(list)
    for path in csv_paths:
        for r in csv.DictReader(open(path)):
            acc[short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in acc.items()}, {k: len(v) for k, v in acc.items()}


def _counter(csv_path: str):
    return _counters([csv_path])


def traffic(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, copy_bytes, out_md, out_json,
            commands) -> None:
    """fetch_csv / write_csv may each list several collections (comma
    separated, one per workload run); a kernel seen in several keeps the
    mean over all its dispatches."""
    fetch, n_fetch = _counters(fetch_csv.split(","))
    write, _ = _counters(write_csv.split(","))
    cf, _ = _counter(copy_fetch_csv)
    cw, _ = _counter(copy_write_csv)
    copy_kib = float(copy_bytes) / 1024.0
    ref_f = cf.get("__amd_rocclr_copyBuffer") or max(cf.values())
    ref_w = cw.get("__amd_rocclr_copyBuffer") or max(cw.values())
    f_scale = copy_kib / ref_f
    w_scale = copy_kib / ref_w
    lines = [f"# HBM traffic per launch (FETCH_SIZE, WRITE_SIZE)", "",
             "Commands:", ""] + [f"    {c}" for c in commands.split(";")] + [
             "", f"Calibration: a {copy_bytes} B device copy reads FETCH_SIZE = {ref_f:.1f} KiB and "
             f"WRITE_SIZE = {ref_w:.1f} KiB per dispatch, so fetch counts are scaled by "
             f"{f_scale:.4f} and write counts by {w_scale:.4f}.", "",
             "| kernel | dispatches | fetch MB | write MB | total MB |", "|---|---:|---:|---:|---:|"]
    per_kernel = {}
    for k in sorted(fetch, key=lambda k: -fetch[k]):
        fb = fetch[k] * f_scale * 1024.0
        wb = write.get(k, 0.0) * w_scale * 1024.0
        per_kernel[k] = {"fetch_bytes": fb, "write_bytes": wb}
        lines.append(f"| `{k}` | {n_fetch[k]} | {fb / 1e6:.2f} | {wb / 1e6:.2f} | {(fb + wb) / 1e6:.2f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")
    lm = {k: v for k, v in per_kernel.items() if "lm_head" in k}
    rec = {"lm_head_source_sha256": lm_head_source_hash(), "fetch_scale": f_scale,
           "write_scale": w_scale, "per_variant": lm, "commands": commands}
    with open(out_json, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")


def counters(csv_path: str, out_md: str, command: str, match: str = "") -> None:
    """Mean of every counter per kernel (kernels whose name contains `match`)."""
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in csv.DictReader(open(csv_path)):
        k = short(r["Kernel_Name"])
        if match in k:
            acc[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    names = sorted({c for v in acc.values() for c in v})
    lines = [f"# Counters per dispatch: `{command}`", "",
             "Means over the dispatches of each kernel (rocprofv3 sums each counter over the",
             "whole device).", "",
             "| kernel | dispatches | " + " | ".join(names) + " |",
             "|---|---:|" + "---:|" * len(names)]
    for k in sorted(acc):
        n = max(len(v) for v in acc[k].values())
        cells = [f"{sum(acc[k][c]) / len(acc[k][c]):.4g}" if acc[k][c] else "" for c in names]
        lines.append(f"| `{k}` | {n} | " + " | ".join(cells) + " |")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


# HIP / HSA calls that load, register or compile code objects
LOADERS = ("hipModuleLoad", "hipModuleLoadData", "hipModuleLoadDataEx", "hipModuleGetFunction",
           "hipModuleUnload", "hiprtc", "__hipRegisterFatBinary", "__hipRegisterFunction",
           "hsa_executable_load_agent_code_object", "hsa_executable_load_program_code_object",
           "hsa_code_object_reader_create_from_memory", "hsa_code_object_reader_create_from_file",
           "hsa_executable_create", "hsa_executable_create_alt", "hsa_executable_freeze",
           "hsa_code_object_deserialize", "hsa_ext_program")


def _api_rows(csv_path):
    out = []
    for r in csv.DictReader(open(csv_path)):
        name = r.get("Function") or r.get("Operation") or r.get("Name") or ""
        out.append((name, int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    return out


def apiwindow(hip_csv: str, hsa_csv: str, out_md: str, command: str) -> None:
    hip = _api_rows(hip_csv)
    hsa = _api_rows(hsa_csv) if hsa_csv and os.path.exists(hsa_csv) else []
    marks = sorted(t0 for n, t0, _ in hip if n == "hipMemGetInfo")
    if len(marks) < 2:
        raise SystemExit("no timed-region markers (hipMemGetInfo) in the HIP trace")
    w0, w1 = marks[-2], marks[-1]
    inside = collections.Counter()
    for n, t0, _ in hip + hsa:
        if w0 < t0 < w1:
            inside[n] += 1
    loads = [(n, t0) for n, t0, _ in hip + hsa if n.startswith(LOADERS)]
    loads_inside = [(n, t0) for n, t0 in loads if w0 < t0 < w1]
    lines = [f"# HIP / HSA API calls in the timed region: `{command}`", "",
             "rocprofv3 --hip-trace --hsa-trace.  The timed region is the interval between the",
             "benchmark's last two hipMemGetInfo calls, made right before the timed steps start",
             "and right after the final synchronisation.", "",
             f"Timed region: {(w1 - w0) / 1e6:.3f} ms.  Code-object load, registration or compile",
             f"calls in the whole run: {len(loads)}; inside the timed region: {len(loads_inside)}.", ""]
    if loads:
        by = collections.Counter(n for n, _ in loads)
        lines += ["| code-object call (whole run) | calls | last call, ms before the timed region |",
                  "|---|---:|---:|"]
        for n, c in sorted(by.items()):
            last = max(t0 for m, t0 in loads if m == n)
            lines.append(f"| `{n}` | {c} | {(w0 - last) / 1e6:.1f} |")
        lines.append("")
    lines += ["| API call inside the timed region | calls |", "|---|---:|"]
    for n, c in sorted(inside.items(), key=lambda kv: -kv[1]):
        lines.append(f"| `{n}` | {c} |")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(sys.argv[2], sys.argv[3], sys.argv[4])
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:10])
    elif sys.argv[1] == "counters":
        counters(*sys.argv[2:6])
    elif sys.argv[1] == "apiwindow":
        apiwindow(*sys.argv[2:6])
    else:
        sys.exit(__doc__)
