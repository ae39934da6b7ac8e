"""Turn rocprofv3 CSV output into the short text summaries kept under
profiles/, and read the counter figures back for bench.py.

    python -m paper_2410_14740_amd.rocprof_summary ffn --name NAME --command CMD \
        --trace DIR/PREFIX_kernel_trace.csv --calls N \
        --fetch DIR/PREFIX_counter_collection.csv --write DIR/PREFIX_counter_collection.csv \
        --copy-fetch ... --copy-write ... --copy-bytes B --out profiles/NAME.md
    python -m paper_2410_14740_amd.rocprof_summary stats --name NAME --command CMD \
        --stats DIR/PREFIX_kernel_stats.csv --out profiles/NAME.md
    python -m paper_2410_14740_amd.rocprof_summary kernels --name NAME --command CMD \
        --kernel NAME1 --kernel NAME2 --trace ... --fetch ... --write ... \
        --copy-fetch ... --copy-write ... --copy-bytes B --algorithmic-bytes A --out profiles/NAME.md
    python -m paper_2410_14740_amd.rocprof_summary counters --name NAME --command CMD \
        --kernel NAME --pmc DIR/PREFIX_counter_collection.csv [--pmc ...] --last N --out profiles/NAME.md

The FFN summary holds the average duration of each sparse-FFN kernel over the
last N back-to-back calls of the trace, the HBM bytes per call from the
FETCH_SIZE and WRITE_SIZE counters (KiB per dispatch) scaled by what the same
counters read for a device copy of known size, and the SHA-256 of the FFN
kernel sources, so that a reader (bench.py) can tell whether the kernels have
changed since the counters were taken.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
FFN_SOURCES = ("csrc/k_ffn_fused.hip", "csrc/ffn_tasks.h", "csrc/ffn_device.h")
FFN_KERNELS = ("ffn_fused_kernel",)


def ffn_source_hash() -> str:
    h = hashlib.sha256()
    for rel in FFN_SOURCES:
        with open(os.path.join(PKG, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _short(name: str) -> str:
    return name.replace("(anonymous namespace)::", "").split("(")[0].replace("void ", "")


def _per_kernel_counter(path: str, kernels) -> dict:
    """Mean counter value (KiB) per dispatch of each named kernel."""
    vals = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        n = _short(r["Kernel_Name"])
        for k in kernels:
            if k in n:
                vals[k].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in vals.items() if v}


def _copy_counter(path: str) -> float:
    """Mean counter value (KiB) per dispatch of the runtime's copy kernel."""
    v = [float(r["Counter_Value"]) for r in csv.DictReader(open(path))
         if "copyBuffer" in r["Kernel_Name"]]
    return sum(v) / len(v)


def ffn_summary(a) -> str:
    rows = [r for r in csv.DictReader(open(a.trace)) if any(k in r["Kernel_Name"] for k in FFN_KERNELS)]
    tail = rows[-len(FFN_KERNELS) * a.calls:]
    dur = collections.defaultdict(list)
    for r in tail:
        dur[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    span = (max(int(r["End_Timestamp"]) for r in tail) - min(int(r["Start_Timestamp"]) for r in tail)) / 1e3
    fetch = _per_kernel_counter(a.fetch, FFN_KERNELS)
    write = _per_kernel_counter(a.write, FFN_KERNELS)
    cf = a.copy_bytes / 1024.0 / _copy_counter(a.copy_fetch)
    cw = a.copy_bytes / 1024.0 / _copy_counter(a.copy_write)
    traffic = sum(fetch.values()) * 1024 * cf + sum(write.values()) * 1024 * cw
    data = {"source_sha256": ffn_source_hash(), "calls": a.calls,
            "us_per_call_span": span / a.calls,
            "kernel_us": {k: sum(v) / len(v) for k, v in dur.items()},
            "fetch_KiB": fetch, "write_KiB": write, "fetch_scale": cf, "write_scale": cw,
            "traffic_bytes_per_call": traffic, "algorithmic_bytes_per_call": a.algorithmic_bytes}
    lines = [f"# {a.name}", "", a.description, "",
             "Commands (from the repository root, on one MI355X):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", "| Kernel | Avg duration (us) | FETCH_SIZE (KiB/dispatch) | WRITE_SIZE (KiB/dispatch) |",
              "|---|---|---|---|"]
    for k in sorted(dur):
        kk = next(x for x in FFN_KERNELS if x in k)
        lines.append(f"| `{k}` | {data['kernel_us'][k]:.2f} | {fetch.get(kk, 0):.1f} | {write.get(kk, 0):.1f} |")
    lines += ["",
              f"* {a.calls} back-to-back calls span {span:.1f} us: {span / a.calls:.2f} us per call.",
              f"* Counter scale from a {a.copy_bytes / 2**20:.0f} MiB device copy: FETCH_SIZE x{cf:.3f}, "
              f"WRITE_SIZE x{cw:.3f}.",
              f"* HBM-side traffic per call: {traffic / 1e6:.2f} MB against {a.algorithmic_bytes / 1e6:.2f} MB "
              f"algorithmic ({traffic / a.algorithmic_bytes:.3f}x).",
              "", "```json", json.dumps(data, indent=1, sort_keys=True), "```", ""]
    return "\n".join(lines)


def kernels_summary(a) -> str:
    """Average duration and HBM-side bytes per dispatch of the named kernels
    (one dispatch of each per step), against the step's algorithmic bytes."""
    names = a.kernel
    dur = collections.defaultdict(list)
    for r in csv.DictReader(open(a.trace)):
        for k in names:
            if k in r["Kernel_Name"]:
                dur[k].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    fetch = _per_kernel_counter(a.fetch, names)
    write = _per_kernel_counter(a.write, names)
    cf = a.copy_bytes / 1024.0 / _copy_counter(a.copy_fetch)
    cw = a.copy_bytes / 1024.0 / _copy_counter(a.copy_write)
    lines = [f"# {a.name}", "", a.description, "",
             "Commands (from the repository root, on one MI355X):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", "| Kernel | Dispatches | Avg duration (us) | FETCH_SIZE (KiB/dispatch) | WRITE_SIZE (KiB/dispatch) "
              "| HBM-side MB/dispatch |", "|---|---|---|---|---|---|"]
    total, total_us = 0.0, 0.0
    for k in names:
        mb = (fetch.get(k, 0.0) * cf + write.get(k, 0.0) * cw) * 1024 / 1e6
        us = sum(dur[k]) / len(dur[k]) if dur[k] else 0.0
        total += mb
        total_us += us
        lines.append(f"| `{k}` | {len(dur[k])} | {us:.2f} | {fetch.get(k, 0.0):.1f} | {write.get(k, 0.0):.1f} "
                     f"| {mb:.2f} |")
    alg = a.algorithmic_bytes / 1e6
    lines += ["",
              f"* Counter scale from a {a.copy_bytes / 2**20:.0f} MiB device copy: FETCH_SIZE x{cf:.3f}, "
              f"WRITE_SIZE x{cw:.3f}.",
              f"* Per step: {total:.2f} MB HBM-side against {alg:.2f} MB algorithmic ({total / alg:.3f}x), "
              f"{total_us:.1f} us in these kernels: {a.algorithmic_bytes / (total_us * 1e3):.0f} GB/s "
              f"algorithmic.", ""]
    return "\n".join(lines)


def counters_summary(a) -> str:
    """Mean value per dispatch of every counter in the given collection files
    (one rocprofv3 --pmc pass each), over the last N dispatches of the named
    kernel, with the ratios that say where its time goes."""
    vals = collections.defaultdict(list)
    for path in a.pmc:
        for r in csv.DictReader(open(path)):
            if a.kernel in r["Kernel_Name"]:
                vals[r["Counter_Name"]].append(float(r["Counter_Value"]))
    mean = {k: sum(v[-a.last:]) / len(v[-a.last:]) for k, v in vals.items() if v}
    lines = [f"# {a.name}", "", a.description, "", "Commands (from the repository root, on one MI355X):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", f"| Counter (`{a.kernel}`, mean of the last {a.last} dispatches) | Value |", "|---|---|"]
    for k in sorted(mean):
        lines.append(f"| `{k}` | {mean[k]:.1f} |")
    derived = {}
    if mean.get("SQ_WAVES"):
        w = mean["SQ_WAVES"]
        for k in ("SQ_INSTS_VALU", "SQ_INSTS_VMEM_RD", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_INSTS_SMEM"):
            if k in mean:
                derived[f"{k} per wave"] = mean[k] / w
    if mean.get("SQ_WAVE_CYCLES"):
        wc = mean["SQ_WAVE_CYCLES"]
        for k in ("SQ_WAIT_INST_ANY", "SQ_WAIT_ANY", "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_ANY"):
            if k in mean:
                derived[f"{k} / SQ_WAVE_CYCLES"] = mean[k] / wc
    if mean.get("TCC_REQ_sum") and "TCC_HIT_sum" in mean:
        derived["L2 hit rate (TCC_HIT / TCC_REQ)"] = mean["TCC_HIT_sum"] / mean["TCC_REQ_sum"]
    if mean.get("GRBM_GUI_ACTIVE") and "SQ_BUSY_CYCLES" in mean:
        derived["SQ_BUSY_CYCLES / GRBM_GUI_ACTIVE"] = mean["SQ_BUSY_CYCLES"] / mean["GRBM_GUI_ACTIVE"]
    if derived:
        lines += ["", "| Derived | Value |", "|---|---|"]
        for k, v in derived.items():
            lines.append(f"| {k} | {v:.3f} |")
    lines += ["", "```json", json.dumps({"kernel": a.kernel, "last": a.last, "mean": mean,
                                         "derived": derived}, indent=1, sort_keys=True), "```", ""]
    return "\n".join(lines)


def stats_summary(a) -> str:
    rows = list(csv.DictReader(open(a.stats)))
    lines = [f"# {a.name}", "", a.description, "", "Command (from the repository root, on one MI355X):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", "| Kernel | Calls | Total (ms) | Average (us) | Min (us) | Max (us) | % of GPU time |",
              "|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| `{_short(r['Name'])}` | {r['Calls']} | {int(r['TotalDurationNs']) / 1e6:.2f} | "
                     f"{float(r['AverageNs']) / 1e3:.2f} | {int(r['MinNs']) / 1e3:.2f} | "
                     f"{int(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(lines) + "\n"


def read_ffn_traffic(path: str):
    """traffic_bytes_per_call from a summary written by ffn_summary, or None
    if the file is missing or the FFN sources have changed since."""
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    data = json.loads(m.group(1))
    if data.get("source_sha256") != ffn_source_hash():
        return None
    return data.get("traffic_bytes_per_call")


def main():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = p.add_subparsers(dest="mode", required=True)
    f = sub.add_parser("ffn")
    for n in ("--trace", "--fetch", "--write", "--copy-fetch", "--copy-write", "--out", "--name"):
        f.add_argument(n, required=True)
    f.add_argument("--calls", type=int, required=True)
    f.add_argument("--copy-bytes", type=int, required=True)
    f.add_argument("--algorithmic-bytes", type=int, required=True)
    f.add_argument("--command", action="append", required=True)
    f.add_argument("--description", default="")
    kp = sub.add_parser("kernels")
    for n in ("--name", "--trace", "--fetch", "--write", "--copy-fetch", "--copy-write", "--out"):
        kp.add_argument(n, required=True)
    kp.add_argument("--kernel", action="append", required=True)
    kp.add_argument("--copy-bytes", type=int, required=True)
    kp.add_argument("--algorithmic-bytes", type=int, required=True)
    kp.add_argument("--command", action="append", required=True)
    kp.add_argument("--description", default="")
    cp = sub.add_parser("counters")
    for n in ("--name", "--kernel", "--out"):
        cp.add_argument(n, required=True)
    cp.add_argument("--pmc", action="append", required=True)
    cp.add_argument("--last", type=int, default=40)
    cp.add_argument("--command", action="append", required=True)
    cp.add_argument("--description", default="")
    s = sub.add_parser("stats")
    for n in ("--stats", "--out", "--name"):
        s.add_argument(n, required=True)
    s.add_argument("--command", action="append", required=True)
    s.add_argument("--description", default="")
    a = p.parse_args()
    text = {"ffn": ffn_summary, "kernels": kernels_summary, "stats": stats_summary,
            "counters": counters_summary}[a.mode](a)
    with open(a.out, "w") as fh:
        fh.write(text)
    print(text)


if __name__ == "__main__":
    main()
