"""Turn rocprofv3 output into the short summaries kept under profiles/.

    python -m paper_2605_01060_amd.profiling stats KERNEL_STATS_CSV --command "..."
    python -m paper_2605_01060_amd.profiling traffic FETCH_CSV WRITE_CSV \
        --kernel-class ffn1 --copy-mib 2048 --command-fetch "..." --command-write "..."

`stats` renders a kernel-trace `*_kernel_stats.csv` as a markdown table.
`mfma` turns a `--pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES` run into
the MFMA-busy share of each kernel class (MFMA busy cycles summed over the
SIMDs / (4 SIMDs x CU busy cycles)).
`clock` turns a `--pmc GRBM_GUI_ACTIVE` run into the engine clock of each
kernel class.
`traffic` reads two `--pmc` runs (FETCH_SIZE, then WRITE_SIZE, KiB per
dispatch), scales each by what the same counter reads for the plain device
copy of known size that the benchmark runs first (`--copy-calibration-mb`),
and reports HBM bytes per launch of one kernel class, together with the
SHA-256 of the kernel's source file so that a stale figure is recognisable.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re
import statistics
import sys
from typing import Dict, List, Optional, Tuple

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)

# kernel class -> (source file, predicate on the demangled kernel name)
# (linear epilogues: 0 bias, 1 bias+GELU, 2 residual, 3 folded LN, 4 folded
# LN + GELU, 5 residual + row statistics, 6 residual LN + row statistics)
KERNEL_CLASSES = {
    "qkv": ("linear.hip", lambda n: "linear_bf16_kernel" in n and _epi(n) in (0, 3)),
    "ffn1": ("linear.hip", lambda n: "linear_bf16_kernel" in n and _epi(n) in (1, 4)),
    "residual": ("linear.hip", lambda n: "linear_bf16_kernel" in n and _epi(n) in (2, 5, 6)),
    "attn": ("attention.hip", lambda n: "attention_varlen_kernel" in n),
    "layernorm": ("rows.hip", lambda n: "layernorm_kernel" in n or "ln_rows_kernel" in n),
}
COPY_KERNEL = "copyBuffer"


def _epi(name: str) -> int:
    """Epilogue of a linear kernel instance: the template argument before
    the tile order (the last one)."""
    m = re.search(r"linear_bf16_kernel<([^>]*)>", name)
    return int(m.group(1).split(",")[-2]) if m else -1


def source_hash(kernel_class: str) -> str:
    fname = KERNEL_CLASSES[kernel_class][0]
    h = hashlib.sha256()
    for f in (fname, "device_common.h"):
        with open(os.path.join(PKG, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stats_markdown(path: str, command: str, top: int = 12) -> str:
    rows = list(csv.DictReader(open(path)))
    out = [f"Command: `{command}`", "", "| kernel | calls | mean µs | total ms | % |",
           "|---|---|---|---|---|"]
    for r in rows[:top]:
        name = r["Name"]
        short = name.replace("surge::(anonymous namespace)::", "").replace("void ", "")
        short = re.sub(r"\(.*", "", short)
        out.append(f"| `{short}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['TotalDurationNs']) / 1e6:.1f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def _per_dispatch(path: str, counter: str) -> Dict[str, List[float]]:
    vals: Dict[str, List[float]] = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return vals


def traffic(fetch_csv: str, write_csv: str, kernel_class: str, copy_mib: float) -> Dict:
    pred = KERNEL_CLASSES[kernel_class][1]
    res = {"kernel_class": kernel_class, "copy_bytes": copy_mib * 2 ** 20,
           "source_sha256": source_hash(kernel_class)}
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"),
                               ("write", write_csv, "WRITE_SIZE")):
        vals = _per_dispatch(path, counter)
        copy = [v for n, vs in vals.items() if COPY_KERNEL in n for v in vs]
        if not copy:
            raise SystemExit(f"no {COPY_KERNEL} dispatch in {path}")
        copy_kib = max(copy)  # the calibration copy is the largest copy dispatch
        scale = (copy_mib * 1024.0) / copy_kib
        ks = [v for n, vs in vals.items() if pred(n) for v in vs]
        if not ks:
            raise SystemExit(f"no {kernel_class} dispatch in {path}")
        res[f"{key}_kib_per_dispatch_raw"] = statistics.fmean(ks)
        res[f"{key}_copy_kib"] = copy_kib
        res[f"{key}_scale"] = scale
        res[f"{key}_bytes_per_launch"] = statistics.fmean(ks) * 1024.0 * scale
        res[f"{key}_dispatches"] = len(ks)
    res["bytes_per_launch"] = res["fetch_bytes_per_launch"] + res["write_bytes_per_launch"]
    return res


def load_traffic(kernel_class: str, workload: str) -> Optional[float]:
    """HBM bytes per launch recorded under profiles/, or None if absent or if
    the kernel's source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}_{workload}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_sha256") != source_hash(kernel_class):
        return None
    return float(rec["bytes_per_launch"])


def mfma_busy(csv_path: str) -> Dict[str, Dict[str, float]]:
    per: Dict[str, Dict[str, float]] = {}
    rows = list(csv.DictReader(open(csv_path)))
    by_dispatch: Dict[Tuple[str, str], Dict[str, float]] = {}
    for r in rows:
        key = (r.get("Dispatch_Id", r.get("Correlation_Id", "")), r["Kernel_Name"])
        by_dispatch.setdefault(key, {})[r["Counter_Name"]] = float(r["Counter_Value"])
    for (_, name), c in by_dispatch.items():
        if "SQ_VALU_MFMA_BUSY_CYCLES" not in c or "SQ_BUSY_CU_CYCLES" not in c:
            continue
        for cls, (_, pred) in KERNEL_CLASSES.items():
            if pred(name):
                e = per.setdefault(cls, {"mfma": 0.0, "busy": 0.0, "dispatches": 0})
                e["mfma"] += c["SQ_VALU_MFMA_BUSY_CYCLES"]
                e["busy"] += c["SQ_BUSY_CU_CYCLES"]
                e["dispatches"] += 1
    return {k: {"mfma_busy_pct": 100.0 * v["mfma"] / (4.0 * v["busy"]) if v["busy"] else 0.0,
                "dispatches": v["dispatches"]} for k, v in per.items()}


def clock(csv_path: str, nominal_ghz: float = 2.4, peak_tflops: float = 2516.6
          ) -> Dict[str, Dict[str, float]]:
    """Mean engine clock of each kernel class from a `--pmc GRBM_GUI_ACTIVE`
    run: the counter is summed over the 8 XCDs, so the clock of a dispatch
    is GRBM_GUI_ACTIVE / 8 / duration.  Also the bf16 MFMA peak at that
    clock (the nominal peak scaled by clock / 2.4 GHz)."""
    per: Dict[str, Dict[str, float]] = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != "GRBM_GUI_ACTIVE":
            continue
        dur = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
        for cls, (_, pred) in KERNEL_CLASSES.items():
            if pred(r["Kernel_Name"]) and dur > 0:
                e = per.setdefault(cls, {"cycles": 0.0, "ns": 0.0, "dispatches": 0})
                e["cycles"] += float(r["Counter_Value"]) / 8.0
                e["ns"] += dur
                e["dispatches"] += 1
    out = {}
    for k, v in per.items():
        ghz = v["cycles"] / v["ns"]
        out[k] = {"dispatches": v["dispatches"], "mean_us": v["ns"] / v["dispatches"] / 1e3,
                  "ghz": ghz, "peak_at_clock_tflops": peak_tflops * ghz / nominal_ghz}
    return out


# bench.py kernel names -> traffic class under profiles/
BENCH_TRAFFIC = {"qkv": "qkv", "ffn1": "ffn1", "oproj": "residual", "ffn2": "residual",
                 "attn": "attn", "ln1": "layernorm", "ln2": "layernorm"}
MFMA_CLASSES = ("qkv", "oproj", "ffn1", "ffn2")


def roofline_markdown(bench_json: str, workload: str, command: str,
                      peak_tflops: float = 2516.6, peak_gbs: float = 8000.0) -> str:
    """Every kernel class of one benchmark line against its own roof: the
    time it would take at the bf16 MFMA peak on its algorithmic FLOPs and at
    the HBM peak on its algorithmic bytes, whichever is longer (the bound),
    with the fraction of that roof achieved, and the measured HBM bytes per
    launch where profiles/ holds a current figure."""
    d = json.load(open(bench_json))
    if d.get("kernels_from"):
        # per-kernel times from one untimed profiled step; the roofline
        # kernel timed again inside the timed region
        src, steps = d["kernels_from"], 1
    else:
        src, steps = "HIP events inside the timed region", d["steps"]
    ridge = peak_tflops * 1e12 / (peak_gbs * 1e9)
    lines = [f"From `{command}` (one JSON line; per-kernel times: {src}) and the traffic "
             f"summaries under `profiles/`.", "",
             f"Value: {d['value']:.0f} texts/s, {d['ms_per_step']:.1f} ms per step, "
             f"MFMA util {d['mfma_util_pct']:.1f} % of {peak_tflops} TFLOP/s."]
    rf = d.get("roofline")
    if rf:
        lines.append(f"Roofline kernel `{rf['kernel']}` in the timed region: "
                     f"{rf['achieved']:.0f} {rf['unit']} of {rf['peak']} "
                     f"(frac {rf['frac']:.3f}), {rf['avg_launch_ms']:.3f} ms per launch.")
    lines += ["",
              f"Roofs: bf16 MFMA {peak_tflops} TFLOP/s, HBM {peak_gbs:.0f} GB/s (ridge "
              f"{ridge:.0f} FLOP/B).  A kernel's roof time is the longer of its algorithmic "
              "FLOPs at the MFMA peak and its algorithmic bytes at the HBM peak.", "",
              "| kernel | launches/step | ms/step | TFLOP/s | GB/s (algorithmic) | FLOP/B | "
              "bound | roof ms/step | % of roof | HBM bytes/launch (measured) | "
              "algorithmic bytes/launch |",
              "|---|---|---|---|---|---|---|---|---|---|---|"]
    tot_ms = tot_roof = 0.0
    for k, v in d["kernels"].items():
        per_launch_bytes = None
        if k in BENCH_TRAFFIC:
            per_launch_bytes = load_traffic(BENCH_TRAFFIC[k], workload)
        ms = v["total_ms_per_step"]
        flops = v.get("tflops", 0.0) * 1e12 * ms / 1e3
        nbytes = v.get("gbs", 0.0) * 1e9 * ms / 1e3
        t_mfma = flops / (peak_tflops * 1e12) * 1e3
        t_hbm = nbytes / (peak_gbs * 1e9) * 1e3
        roof = max(t_mfma, t_hbm)
        bound = "mfma" if t_mfma >= t_hbm else "hbm"
        ai = flops / nbytes if nbytes else float("inf")
        tot_ms += ms
        tot_roof += roof
        alg_bytes = nbytes / v["launches"] * steps if nbytes else None
        lines.append(
            f"| {k} | {v['launches'] / steps:.0f} | {ms:.1f} | {v.get('tflops', 0.0):.0f} | "
            f"{v.get('gbs', 0.0):.0f} | {ai:.0f} | {bound} | {roof:.1f} | "
            f"{100 * roof / ms if ms else 0.0:.1f} | "
            f"{'%.3g' % per_launch_bytes if per_launch_bytes else '—'} | "
            f"{'%.3g' % alg_bytes if alg_bytes else '—'} |")
    lines += ["", f"Sum over kernels: {tot_ms:.1f} ms per step against {tot_roof:.1f} ms of "
                  f"roof time ({100 * tot_roof / tot_ms:.1f} % of roof)."]
    return "\n".join(lines) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("csv")
    a.add_argument("--command", required=True)
    r = sub.add_parser("roofline")
    r.add_argument("bench_json")
    r.add_argument("--workload", default="bge")
    r.add_argument("--command", required=True)
    c = sub.add_parser("mfma")
    c.add_argument("csv")
    c.add_argument("--command", required=True)
    k = sub.add_parser("clock")
    k.add_argument("csv")
    k.add_argument("--command", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_csv")
    b.add_argument("write_csv")
    b.add_argument("--kernel-class", required=True, choices=sorted(KERNEL_CLASSES))
    b.add_argument("--copy-mib", type=float, required=True)
    b.add_argument("--command-fetch", required=True)
    b.add_argument("--command-write", required=True)
    args = ap.parse_args(argv)
    if args.cmd == "stats":
        sys.stdout.write(stats_markdown(args.csv, args.command))
    elif args.cmd == "roofline":
        sys.stdout.write(roofline_markdown(args.bench_json, args.workload, args.command))
    elif args.cmd == "mfma":
        res = mfma_busy(args.csv)
        lines = [f"Command: `{args.command}`", "",
                 "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (4 SIMDs x SQ_BUSY_CU_CYCLES), summed "
                 "over the dispatches of each kernel class.", "",
                 "| kernel class | dispatches | MFMA busy % |", "|---|---|---|"]
        for k in sorted(res):
            lines.append(f"| {k} | {res[k]['dispatches']} | {res[k]['mfma_busy_pct']:.1f} |")
        sys.stdout.write("\n".join(lines) + "\n")
    elif args.cmd == "clock":
        res = clock(args.csv)
        lines = [f"Command: `{args.command}`", "",
                 "Engine clock per kernel class = GRBM_GUI_ACTIVE (summed over the 8 XCDs) "
                 "/ 8 / dispatch duration, averaged over the dispatches; the bf16 MFMA peak "
                 "at that clock is 2516.6 TFLOP/s x clock / 2.4 GHz.", "",
                 "| kernel class | dispatches | mean duration us | clock GHz | "
                 "bf16 peak at that clock TFLOP/s |", "|---|---|---|---|---|"]
        for k in sorted(res):
            r = res[k]
            if r["mean_us"] < 50.0:  # counter read-out dominates a short dispatch
                lines.append(f"| {k} | {r['dispatches']} | {r['mean_us']:.1f} | — | — |")
            else:
                lines.append(f"| {k} | {r['dispatches']} | {r['mean_us']:.1f} | "
                             f"{r['ghz']:.3f} | {r['peak_at_clock_tflops']:.0f} |")
        lines += ["", "(Dispatches shorter than 50 us: the counter read-out around the "
                      "dispatch dominates, so no clock is given.)"]
        sys.stdout.write("\n".join(lines) + "\n")
    else:
        rec = traffic(args.fetch_csv, args.write_csv, args.kernel_class, args.copy_mib)
        sys.stdout.write(
            f"HBM traffic of the `{args.kernel_class}` kernel class (mean per launch), from\n\n"
            f"- `{args.command_fetch}`\n- `{args.command_write}`\n\n"
            "Each counter is scaled by what it reads for the benchmark's calibration copy "
            f"({args.copy_mib:.0f} MiB device-to-device, the `{COPY_KERNEL}` dispatch).\n\n"
            f"```json\n{json.dumps(rec, indent=1)}\n```\n")


if __name__ == "__main__":
    main()
