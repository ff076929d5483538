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
`fabric` turns a `--pmc` run of the L2 read-request counters split by
request size into exact L2-to-fabric read bytes per launch of each class.
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

# kernel class -> source file of its kernel
KERNEL_SOURCES = {"qkv": "linear.hip", "oproj": "linear.hip", "ffn1": "linear.hip",
                  "ffn2": "linear.hip", "attn": "attention.hip", "layernorm": "rows.hip"}
KERNEL_CLASSES = tuple(KERNEL_SOURCES)
COPY_KERNEL = "copyBuffer"


def _epi(name: str) -> int:
    """Epilogue of a linear kernel instance: the template argument before
    the tile order (the last one)."""
    m = re.search(r"linear_bf16_kernel<([^>]*)>", name)
    return int(m.group(1).split(",")[-2]) if m else -1


def name_class(name: str) -> Optional[str]:
    """Kernel class from the demangled name alone (linear epilogues: 0 bias,
    1 bias+GELU, 2 residual, 3 folded LN, 4 folded LN + GELU, 5 residual +
    row statistics, 6 residual LN + row statistics).  The O-projection and
    FFN2 run the same residual-epilogue instance and come back as
    "residual"; `dispatch_classes` tells them apart."""
    if "linear_bf16_kernel" in name:
        return {0: "qkv", 3: "qkv", 1: "ffn1", 4: "ffn1",
                2: "residual", 5: "residual", 6: "residual"}.get(_epi(name))
    if "attention_varlen_kernel" in name:
        return "attn"
    if "layernorm_kernel" in name or "ln_rows_kernel" in name:
        return "layernorm"
    return None


def dispatch_classes(names: List[str]) -> List[Optional[str]]:
    """Kernel class of every dispatch, given the names in dispatch order: a
    residual-epilogue GEMM is FFN2 when the linear dispatch before it was
    FFN1 (the FFN output), and the O-projection otherwise."""
    out: List[Optional[str]] = []
    last_linear = None
    for n in names:
        c = name_class(n)
        if c == "residual":
            c = "ffn2" if last_linear == "ffn1" else "oproj"
        if c in ("qkv", "ffn1", "oproj", "ffn2"):
            last_linear = c
        out.append(c)
    return out


def _dispatches(path: str) -> List[Dict]:
    """The dispatches of a counter-collection CSV in dispatch order, each
    with its name, class, duration (ns, where timestamps are present) and
    counters."""
    by_id: Dict[int, Dict] = {}
    for r in csv.DictReader(open(path)):
        key = int(r.get("Dispatch_Id") or r.get("Correlation_Id"))
        e = by_id.setdefault(key, {"name": r["Kernel_Name"], "counters": {}, "ns": 0.0})
        e["counters"][r["Counter_Name"]] = (e["counters"].get(r["Counter_Name"], 0.0)
                                            + float(r["Counter_Value"]))
        if r.get("Start_Timestamp") and r.get("End_Timestamp"):
            e["ns"] = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
    disp = [by_id[k] for k in sorted(by_id)]
    for e, c in zip(disp, dispatch_classes([e["name"] for e in disp])):
        e["cls"] = c
    return disp


def source_hash(kernel_class: str) -> str:
    fname = KERNEL_SOURCES[kernel_class]
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


def traffic(fetch_csv: str, write_csv: str, kernel_class: str, copy_mib: float) -> Dict:
    res = {"kernel_class": kernel_class, "copy_bytes": copy_mib * 2 ** 20,
           "source_sha256": source_hash(kernel_class)}
    for key, path, counter in (("fetch", fetch_csv, "FETCH_SIZE"),
                               ("write", write_csv, "WRITE_SIZE")):
        disp = [e for e in _dispatches(path) if counter in e["counters"]]
        copy = [e["counters"][counter] for e in disp if COPY_KERNEL in e["name"]]
        if not copy:
            raise SystemExit(f"no {COPY_KERNEL} dispatch in {path}")
        copy_kib = max(copy)  # the calibration copy is the largest copy dispatch
        scale = (copy_mib * 1024.0) / copy_kib
        ks = [e["counters"][counter] for e in disp if e["cls"] == kernel_class]
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
    for e in _dispatches(csv_path):
        c = e["counters"]
        if e["cls"] is None or "SQ_VALU_MFMA_BUSY_CYCLES" not in c or "SQ_BUSY_CU_CYCLES" not in c:
            continue
        v = per.setdefault(e["cls"], {"mfma": 0.0, "busy": 0.0, "dispatches": 0})
        v["mfma"] += c["SQ_VALU_MFMA_BUSY_CYCLES"]
        v["busy"] += c["SQ_BUSY_CU_CYCLES"]
        v["dispatches"] += 1
    return {k: {"mfma_busy_pct": 100.0 * v["mfma"] / (4.0 * v["busy"]) if v["busy"] else 0.0,
                "dispatches": v["dispatches"]} for k, v in per.items()}


def clock(csv_path: str, nominal_ghz: float = 2.4, peak_tflops: float = 2516.6
          ) -> Dict[str, Dict[str, float]]:
    """Mean engine clock of each kernel class from a `--pmc GRBM_GUI_ACTIVE`
    run: the counter is summed over the 8 XCDs, so the clock of a dispatch
    is GRBM_GUI_ACTIVE / 8 / duration.  Also the bf16 MFMA peak at that
    clock (the nominal peak scaled by clock / 2.4 GHz)."""
    per: Dict[str, Dict[str, float]] = {}
    for e in _dispatches(csv_path):
        if e["cls"] is None or "GRBM_GUI_ACTIVE" not in e["counters"] or e["ns"] <= 0:
            continue
        v = per.setdefault(e["cls"], {"cycles": 0.0, "ns": 0.0, "dispatches": 0})
        v["cycles"] += e["counters"]["GRBM_GUI_ACTIVE"] / 8.0
        v["ns"] += e["ns"]
        v["dispatches"] += 1
    out = {}
    for k, v in per.items():
        ghz = v["cycles"] / v["ns"]
        out[k] = {"dispatches": v["dispatches"], "mean_us": v["ns"] / v["dispatches"] / 1e3,
                  "ghz": ghz, "peak_at_clock_tflops": peak_tflops * ghz / nominal_ghz}
    return out


READ_SIZES = {"TCC_EA0_RDREQ_128B_sum": 128.0, "TCC_EA0_RDREQ_64B_sum": 64.0,
              "TCC_EA0_RDREQ_32B_sum": 32.0}


def fabric_reads(csv_path: str) -> Dict[str, Dict[str, float]]:
    """L2-to-fabric read bytes per launch of each kernel class from a `--pmc
    TCC_EA0_RDREQ_128B_sum TCC_EA0_RDREQ_64B_sum TCC_EA0_RDREQ_32B_sum
    TCC_EA0_RDREQ_sum` run: every request counted at its own size, so no
    calibration copy is needed (FETCH_SIZE's expression takes 128-byte
    requests from TCC_BUBBLE, which reads 0 on gfx950, and counts them as
    64 bytes).  `accounted` is the share of all read requests that the three
    size classes cover."""
    per: Dict[str, Dict[str, float]] = {}
    for e in _dispatches(csv_path):
        c = e["counters"]
        if e["cls"] is None or not all(k in c for k in READ_SIZES):
            continue
        v = per.setdefault(e["cls"], {"bytes": 0.0, "sized": 0.0, "all": 0.0, "dispatches": 0})
        v["bytes"] += sum(c[k] * b for k, b in READ_SIZES.items())
        v["sized"] += sum(c[k] for k in READ_SIZES)
        v["all"] += c.get("TCC_EA0_RDREQ_sum", 0.0)
        v["dispatches"] += 1
    return {k: {"dispatches": v["dispatches"], "read_bytes_per_launch": v["bytes"] / v["dispatches"],
                "accounted": v["sized"] / v["all"] if v["all"] else float("nan")}
            for k, v in per.items()}


def _stored_fetch(kernel_class: str, workload: str) -> Optional[float]:
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}_{workload}.md")
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    return float(json.loads(m.group(1))["fetch_bytes_per_launch"]) if m else None


# bench.py kernel names -> traffic class under profiles/
BENCH_TRAFFIC = {"qkv": "qkv", "ffn1": "ffn1", "oproj": "oproj", "ffn2": "ffn2",
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
    f = sub.add_parser("fabric")
    f.add_argument("csv")
    f.add_argument("--workload", default="bge")
    f.add_argument("--command", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_csv")
    b.add_argument("write_csv")
    b.add_argument("--kernel-class", required=True, choices=sorted(KERNEL_SOURCES))
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
    elif args.cmd == "fabric":
        res = fabric_reads(args.csv)
        lines = [f"Command: `{args.command}`", "",
                 "L2-to-fabric read bytes per launch = 128 x TCC_EA0_RDREQ_128B + 64 x "
                 "TCC_EA0_RDREQ_64B + 32 x TCC_EA0_RDREQ_32B (summed over the L2 channels and "
                 "XCDs), averaged over the dispatches of each kernel class; beside it the "
                 "copy-calibrated FETCH_SIZE figure of the `traffic_*` summaries.", "",
                 "| kernel class | dispatches | read bytes/launch (request sizes) | "
                 "FETCH_SIZE x calibration | requests covered by the size classes |",
                 "|---|---|---|---|---|"]
        for k in sorted(res):
            r = res[k]
            fs = _stored_fetch(k, args.workload)
            lines.append(f"| {k} | {r['dispatches']} | {r['read_bytes_per_launch']:.4g} | "
                         f"{'%.4g' % fs if fs else '—'} | {100 * r['accounted']:.2f} % |")
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
