"""Benchmark: SuperBatch encoding throughput on one MI355X.

A step is one pass of the whole encode path (SuperBatch formation, packing
metadata, embedding, every encoder layer, pooling, L2 and partition scatter)
over the whole synthetic workload, via surge_encode_all with inputs already
resident in HBM.  Prints one JSON line.

Timing: W untimed warm-up steps; one more untimed step with HIP events
around every kernel launch gives the per-kernel breakdown (`kernels`) and
names the dominant kernel class; then K timed steps between two stream
events, with HIP events recorded only around the dominant class's launches
(its `roofline` figure), so the other launches run back to back.

    python bench.py [--steps K] [--warmup W] [--workload bge] [--gpus 1]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2605_01060_amd import profiling  # noqa: E402
from paper_2605_01060_amd import surge as S  # noqa: E402
from paper_2605_01060_amd import workload as W  # noqa: E402

METRIC = "texts/sec + MFMA util % on 1 MI355X, bge-base-shaped encoder, σ=1.72 parts"
PEAK_BF16_TFLOPS = 2516.6  # 256 CU x 4096 FLOP/clk x 2.4 GHz, dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
MFMA_KERNELS = ("qkv", "oproj", "ffn1", "ffn2")

DESCRIPTIONS = {
    "tiny": "tiny encoder (2 L, d 128), 1,000 texts / 20 partitions, sigma 1.72, B_min 1,000",
    "minilm": "MiniLM-L6-shaped encoder (6 L, d 384), 100k texts / 400 partitions, sigma 1.72, "
              "B_min 4,096, n_max 20,000",
    "bge": "bge-base-shaped encoder (12 L, d 768, 12 H, FFN 3072), 200k texts / 800 partitions, "
           "partition sizes log-normal sigma 1.72, lengths log-normal median 48 in [4, 256], "
           "B_min 4,096, n_max 20,000",
    "bge_s1": "bge-base-shaped encoder, 200k texts / 800 partitions, sigma 1.0, B_min 4,096, "
              "n_max 20,000",
    "minilm_heavy": "MiniLM-L6-shaped encoder, 1M texts / 4,000 partitions, sigma 2.5, "
                    "B_min 8,192, n_max 50,000",
    "large": "~335M encoder (24 L, d 1024), 100k texts / 400 partitions, sigma 1.72, "
             "B_min 2,048, n_max 10,000",
}


def encoder_flops(shape: W.EncoderShape, lengths: np.ndarray) -> float:
    """Algorithmic matmul FLOPs: per text n_layers [2 L (4 d^2 + 2 d d_ff) + 4 d L^2]
    (QKV, O, FFN1, FFN2, Q K^T, P V over the text's own tokens and pairs)."""
    L = lengths.astype(np.float64)
    d, f = shape.d_model, shape.d_ff
    return float(shape.n_layers * (2.0 * L * (4 * d * d + 2 * d * f) + 4.0 * d * L * L).sum())


# Fixed prefix of SuperBatch 0 timed on the host per workload (texts).
CPU_SAMPLE = {"tiny": 1000, "minilm": 2000, "minilm_heavy": 2000, "bge": 1000, "bge_s1": 1000,
              "large": 200}


def host_description():
    """What the CPU baseline ran on: logical CPUs, the CPU model and the
    NumPy BLAS build with the thread count it uses."""
    info = {"nproc": os.cpu_count(), "affinity": len(os.sched_getaffinity(0))}
    try:
        with open("/proc/cpuinfo") as f:
            info["cpu_model"] = next((l.split(":", 1)[1].strip() for l in f
                                      if l.startswith("model name")), None)
    except OSError:
        info["cpu_model"] = None
    try:
        blas = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        info["numpy_blas"] = f"{blas.get('name')} {blas.get('version')}"
    except Exception:
        info["numpy_blas"] = None
    try:
        from threadpoolctl import threadpool_info
        pools = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        info["blas_threads"] = max([p.get("num_threads", 1) for p in pools] + [1])
        info["blas_runtime"] = ", ".join(f"{p.get('internal_api')} {p.get('version')} "
                                         f"({p.get('architecture')})" for p in pools) or None
    except Exception:
        info["blas_threads"] = None
        info["blas_runtime"] = None
    return info


def cpu_baseline(spec, wl, weights, n_sample: int, n_sb0: int):
    """The float32 oracle, as it stands, on the first n_sample texts of
    SuperBatch 0 (one text at a time, every BLAS thread of the host)."""
    from oracle import encoder as E
    host = host_description()
    sh = spec.encoder
    w32 = E.as_f32(weights)
    n = min(n_sample, n_sb0, wl.n_texts)
    toks = int(wl.cu_seqlens[n] - wl.cu_seqlens[0])
    t0 = time.perf_counter()
    E.encode_texts(w32, sh.n_layers, sh.n_heads, wl.tokens, wl.cu_seqlens, range(n), sh.ln_eps)
    dt = time.perf_counter() - t0
    flops = encoder_flops(sh, wl.lengths[:n])
    return {"value": n / dt, "unit": "texts/s", "cores": host["blas_threads"] or host["nproc"],
            "kind": "oracle",
            "sample": f"first {n} texts ({toks} tokens) of SuperBatch 0 of the same workload, "
                      f"float32 NumPy oracle, one text at a time, {dt:.1f} s",
            "tokens_per_s": toks / dt, "gflops": flops / dt / 1e9,
            "extrapolated_full_workload_s": dt * wl.n_texts / n,
            "host": host}


def blas_reference(spec, wl, iters: int = 20):
    """Vendor GEMM (torch.mm, i.e. hipBLASLt) beside the library's own GEMM
    with a bias-only epilogue on the encoder's four projection shapes, at
    the mean SuperBatch token count, on random bf16 data.  Context for the
    GEMM rooflines only: the encode path never calls a library GEMM."""
    import torch
    sh = spec.encoder
    sbs, _ = S.surge_plan(wl.part_offsets, spec.b_min, spec.n_max)
    cu = wl.cu_seqlens
    toks = [int(cu[int(b["text_end"])] - cu[int(b["text_begin"])]) for b in sbs]
    M = int(round(sum(toks) / len(toks)))
    d, f = sh.d_model, sh.d_ff
    shapes = [("qkv", 3 * d, d), ("oproj", d, d), ("ffn1", f, d), ("ffn2", d, f)]
    g = torch.Generator(device="cuda").manual_seed(0)
    out = []
    for name, N, K in shapes:
        x = torch.randn(M, K, device="cuda", generator=g).to(torch.bfloat16)
        w = (torch.randn(N, K, device="cuda", generator=g) * 0.03).to(torch.bfloat16)
        wt = w.t().contiguous()
        b = torch.zeros(N, device="cuda")
        y = torch.empty(M, N, device="cuda", dtype=torch.bfloat16)
        stream = torch.cuda.current_stream()

        def vendor():
            torch.mm(x, wt, out=y)

        def own():
            S.surge_op_linear(M, N, K, x, w, b, None, 0, y, stream)

        row = {"gemm": name, "M": M, "N": N, "K": K}
        for tag, fn in (("hipblaslt_mm", vendor), ("surge_bias_only", own)):
            for _ in range(5):
                fn()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record(stream)
            for _ in range(iters):
                fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / iters
            row[tag + "_ms"] = ms
            row[tag + "_tflops"] = 2.0 * M * N * K / (ms / 1e3) / 1e12
        out.append(row)
        del x, w, wt, b, y
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="bge", choices=sorted(W.WORKLOADS))
    ap.add_argument("--chunk-tokens", type=int, default=1 << 20)
    ap.add_argument("--cpu-texts", type=int, default=0,
                    help="texts of the CPU-oracle sample (default: the workload's fixed prefix)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-events", action="store_true")
    ap.add_argument("--no-stream", action="store_true",
                    help="skip the streamed pass (host tokens in, host embeddings out)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="run one plain device-to-device copy of this many MiB before the "
                         "warm-up (reference for FETCH_SIZE / WRITE_SIZE counter runs)")
    ap.add_argument("--blas-reference", action="store_true",
                    help="only time the vendor GEMM beside the library GEMM on the "
                         "encoder's projection shapes and print them")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(json.dumps({"error": "this path runs on one GPU; --gpus must be 1 "
                                   "(SuperBatches shard across GPUs with no exchange step, "
                                   "but multi-GPU runs are not part of this build)"}))
        return 2

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    spec = W.WORKLOADS[args.workload]
    sh = spec.encoder
    wl = W.make_workload(spec)
    if args.blas_reference:
        print(json.dumps({"workload": args.workload,
                          "blas_reference": blas_reference(spec, wl)}), flush=True)
        return 0
    weights = W.make_weights(sh, seed=spec.seed)
    desc = S.make_desc(sh.n_layers, sh.d_model, sh.n_heads, sh.d_ff, sh.vocab_size,
                       sh.max_positions, sh.ln_eps)
    enc = S.Encoder(desc, [weights[n] for n in W.weight_names(sh.n_layers)], args.chunk_tokens)
    tok = torch.from_numpy(wl.tokens).cuda()
    out = torch.empty((wl.n_texts, sh.d_model), dtype=torch.float32, device="cuda")
    ptrs = np.array([out.data_ptr() + int(o) * sh.d_model * 4 for o in wl.part_offsets[:-1]],
                    dtype=np.uint64)
    stream = torch.cuda.current_stream()
    flops = encoder_flops(sh, wl.lengths)
    if args.copy_calibration_mb > 0:
        n = args.copy_calibration_mb << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    def step():
        return enc.encode_all(wl.n_texts, tok, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                              spec.n_max, ptrs, stream=stream)

    for _ in range(args.warmup):
        n_sb = step()
    enc.check(stream)
    torch.cuda.synchronize()
    print(f"[bench] workload={args.workload} texts={wl.n_texts} tokens={wl.n_tokens} "
          f"warmup done", file=sys.stderr, flush=True)

    # Per-kernel breakdown: one untimed step with events around every launch.
    # The timed steps then record events only around the launches of the
    # dominant kernel class (its roofline figure), so the other launches run
    # back to back as they do without profiling.
    kall = {}
    dom = None
    if not args.no_kernel_events:
        enc.profile(True)
        step()
        kall = enc.profile_read()
        enc.profile(False)
        dom = max(kall, key=lambda k: kall[k]["total_ms"])
        enc.profile(True, kinds=[dom])
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        n_sb = step()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    enc.check(stream)
    kstats = enc.profile_read() if dom is not None else {}
    enc.profile(False)

    ms_step = ms / args.steps
    texts_s = wl.n_texts / (ms_step / 1e3)
    tflops = flops / (ms_step / 1e3) / 1e12
    kernels = {}
    for name, s in kall.items():
        if s["launches"] == 0:
            continue
        avg = s["total_ms"] / s["launches"]
        ent = {"launches": s["launches"], "total_ms_per_step": s["total_ms"], "avg_ms": avg}
        if s["flops"] > 0:
            ent["tflops"] = s["flops"] / (s["total_ms"] / 1e3) / 1e12
        if s["bytes"] > 0:
            ent["gbs"] = s["bytes"] / (s["total_ms"] / 1e3) / 1e9
        kernels[name] = ent
    roofline = None
    if dom is not None and kstats[dom]["launches"] > 0:
        s = kstats[dom]
        traffic = None
        if dom in profiling.BENCH_TRAFFIC:
            traffic = profiling.load_traffic(profiling.BENCH_TRAFFIC[dom], args.workload)
        if dom in MFMA_KERNELS:
            achieved = s["flops"] / (s["total_ms"] / 1e3) / 1e12
            roofline = {"kernel": dom, "bound": "mfma", "achieved": achieved,
                        "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                        "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic,
                        "per_launch_flops": s["flops"] / s["launches"],
                        "per_launch_algorithmic_bytes": s["bytes"] / s["launches"],
                        "avg_launch_ms": s["total_ms"] / s["launches"]}
        else:
            achieved = s["bytes"] / (s["total_ms"] / 1e3) / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": achieved,
                        "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                        "traffic": traffic, "per_launch_bytes": s["bytes"] / s["launches"],
                        "avg_launch_ms": s["total_ms"] / s["launches"]}

    # Streamed pass, outside the timed region: tokens start in pinned host
    # memory and embeddings end there, so PCIe is included.  The reported
    # rate is the zero-copy mode (the pooling kernel writes the pinned output
    # directly, so no download runs); beside it the copies overlapped on a
    # second stream and everything in order on one stream.
    streamed = None
    if not args.no_stream:
        h_tok = torch.from_numpy(wl.tokens).pin_memory()
        h_out = torch.empty((wl.n_texts, sh.d_model), dtype=torch.float32).pin_memory()
        cs, xs = torch.cuda.Stream(), torch.cuda.Stream()
        times = np.zeros((n_sb, 3), np.float64)
        st1 = enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets,
                                      spec.b_min, spec.n_max, h_out, overlap=1,
                                      compute_stream=cs, copy_stream=xs, sb_times=times)
        st0 = enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets,
                                      spec.b_min, spec.n_max, h_out, overlap=0,
                                      compute_stream=cs)
        st2 = enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets,
                                      spec.b_min, spec.n_max, h_out, overlap=2,
                                      compute_stream=cs)
        enc_sb = times[:, 1]
        streamed = {
            "value": wl.n_texts / (st2["total_ms"] / 1e3), "unit": "texts/s",
            "mode": "zero copy (overlap=2): tokens uploaded in order, embeddings written "
                    "into pinned host memory by the pooling kernel",
            "total_ms": st2["total_ms"], "ttfo_ms": st2["ttfo_ms"], "enc_ms": st2["enc_ms"],
            "h2d_ms": st2["h2d_ms"],
            "staging_bytes": st2["staging_bytes"], "max_sb_texts": st2["max_sb_texts"],
            "max_sb_tokens": st2["max_sb_tokens"],
            "overlapped_value": wl.n_texts / (st1["total_ms"] / 1e3),
            "overlapped_total_ms": st1["total_ms"], "overlapped_ttfo_ms": st1["ttfo_ms"],
            "overlapped_h2d_ms": st1["h2d_ms"], "overlapped_d2h_ms": st1["d2h_ms"],
            "overlapped_rho": st1["rho"], "overlapped_rho_measured": st1["rho_measured"],
            "overlapped_staging_bytes": st1["staging_bytes"],
            "sync_value": wl.n_texts / (st0["total_ms"] / 1e3),
            "sync_total_ms": st0["total_ms"], "sync_ttfo_ms": st0["ttfo_ms"],
            "sync_rho_measured": st0["rho_measured"],
            "superbatch_encode_ms": {"n": int(enc_sb.size), "min": float(enc_sb.min()),
                                     "median": float(np.median(enc_sb)),
                                     "max": float(enc_sb.max())},
        }
        print(f"[bench] streamed pass done", file=sys.stderr, flush=True)
        del h_tok, h_out

    cpu = None
    if not args.no_cpu_baseline:
        sbs, _ = S.surge_plan(wl.part_offsets, spec.b_min, spec.n_max)
        n_sb0 = int(sbs[0]["text_end"] - sbs[0]["text_begin"])
        cpu = cpu_baseline(spec, wl, weights, args.cpu_texts or CPU_SAMPLE[args.workload], n_sb0)
        print(f"[bench] cpu baseline done", file=sys.stderr, flush=True)

    line = {
        "metric": METRIC,
        "value": texts_s,
        "unit": "texts/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded workload and random-init weights of the named shape)",
        "config": {"workload": DESCRIPTIONS[args.workload], "name": args.workload,
                   "n_texts": wl.n_texts, "n_tokens": wl.n_tokens, "n_superbatches": n_sb,
                   "chunk_tokens": args.chunk_tokens},
        "tokens_per_s": wl.n_tokens / (ms_step / 1e3),
        "encoder_tflops": tflops,
        "mfma_util_pct": 100.0 * tflops / PEAK_BF16_TFLOPS,
        "kernels": kernels,
        "kernels_from": "one untimed step with HIP events around every launch",
        "roofline": roofline,
        "cpu_baseline": cpu,
        "pcie_inclusive": streamed,
    }
    print(json.dumps(line), flush=True)
    enc.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
