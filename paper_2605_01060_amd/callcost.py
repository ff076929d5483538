"""Per-call cost of the encode path and the IPC-amortization model (Theorem 1).

    python -m paper_2605_01060_amd.callcost [--workload bge] [--bmin 512,1024,...]

The paper's cost model (Sec. 2.3, Theorem 1) charges every encode call a fixed
overhead c_call on top of a per-text cost c_enc, so a plan with F calls over N
texts takes F c_call + N c_enc (one GPU).  On the MI355X the fixed part of a
call is the launch and metadata cost of its ~90 kernels plus the floor that a
small call puts on every GEMM (a launch with fewer tiles than CUs takes as
long as one tile).  This tool runs the same kernels under three plans through
the C-ABI (surge_plan / surge_encode_superbatch):

* PBP: one call per partition (Sec. 2.2);
* FSB: fixed chunks of B texts, cut across partition boundaries (Sec. 2.2);
  the scatter writes each row into its partition, so no regrouping pass is
  needed here;
* SURGE: the two-threshold SuperBatches (Alg. 1, reading R2);

times every call with stream events, fits T(n) = c_call + n c_enc to the PBP
calls (least squares over texts per call), and compares the measured PBP /
SURGE time ratio with Theorem 1's prediction (1 + a) / (1 + a F / P),
a = P c_call / (N c_enc).  A B_min sweep of the SURGE plan shows where
throughput saturates against SuperBatch size (cf. Tab. 7).
"""
from __future__ import annotations

import argparse
import json
import sys
from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import surge as S
from . import workload as W

# A call: (text_begin, text_end, segments with SuperBatch-local first_text).
Call = Tuple[int, int, np.ndarray]


def _calls_from_plan(sbs: np.ndarray, segs: np.ndarray) -> List[Call]:
    out = []
    for sb in sbs:
        g = segs[int(sb["seg_begin"]):int(sb["seg_end"])].copy()
        g["first_text"] -= sb["text_begin"]
        out.append((int(sb["text_begin"]), int(sb["text_end"]), g))
    return out


def plan_pbp(part_offsets: Sequence[int]) -> List[Call]:
    """One call per non-empty partition: the planner with B_min = 1 and no cap."""
    sbs, segs = S.surge_plan(part_offsets, 1, 0, S.SURGE_POLICY_SPLIT)
    return _calls_from_plan(sbs, segs)


def plan_surge(part_offsets: Sequence[int], b_min: int, n_max: int,
               policy: int = S.SURGE_POLICY_SPLIT) -> List[Call]:
    sbs, segs = S.surge_plan(part_offsets, b_min, n_max, policy)
    return _calls_from_plan(sbs, segs)


def plan_fsb(part_offsets: Sequence[int], chunk: int) -> List[Call]:
    """Chunks [kB, (k+1)B) of the concatenated texts; each chunk's segments
    are its intersections with the partitions."""
    offs = np.asarray(part_offsets, np.int64)
    n = int(offs[-1])
    out = []
    for t0 in range(0, n, chunk):
        t1 = min(n, t0 + chunk)
        p0 = int(np.searchsorted(offs, t0, side="right")) - 1
        rows = []
        p = p0
        while p < len(offs) - 1 and offs[p] < t1:
            a, b = max(t0, int(offs[p])), min(t1, int(offs[p + 1]))
            if b > a:
                rows.append((a - t0, b - a, p, a - int(offs[p])))
            p += 1
        out.append((t0, t1, S.segments_array(rows)))
    return out


def ffd_batches(sizes: Sequence[int], capacity: int) -> List[List[int]]:
    """PB-PBP-LB (Sec. 5, stronger baseline): partitions sorted by size,
    largest first (index breaks ties), each packed whole into the first batch
    with room for it, else a new batch."""
    order = sorted((p for p in range(len(sizes)) if sizes[p] > 0), key=lambda p: (-sizes[p], p))
    batches: List[List[int]] = []
    room: List[int] = []
    for p in order:
        n = int(sizes[p])
        for b, r in enumerate(room):
            if n <= r:
                batches[b].append(p)
                room[b] = r - n
                break
        else:
            batches.append([p])
            room.append(capacity - n)
    return batches


def plan_ffd(part_offsets: Sequence[int], cu_seqlens: Sequence[int],
             capacity: int) -> Tuple[List[Call], np.ndarray, np.ndarray]:
    """FFD batches as calls.  A batch's partitions are not adjacent in the
    input, so the texts are re-laid out batch after batch: returns the calls
    over that layout, the text permutation (new position -> original text)
    and the layout's cu_seqlens.  Rows still go to the original partitions
    (segments name the partition, row offset 0)."""
    offs = np.asarray(part_offsets, np.int64)
    cu = np.asarray(cu_seqlens, np.int64)
    sizes = np.diff(offs)
    perm_parts: List[int] = []
    calls: List[Call] = []
    t0 = 0
    for batch in ffd_batches(sizes, capacity):
        rows = []
        local = 0
        for p in batch:
            rows.append((local, int(sizes[p]), p, 0))
            local += int(sizes[p])
            perm_parts.append(p)
        calls.append((t0, t0 + local, S.segments_array(rows)))
        t0 += local
    perm = (np.concatenate([np.arange(offs[p], offs[p + 1]) for p in perm_parts])
            if perm_parts else np.zeros(0, np.int64))
    lens = (cu[1:] - cu[:-1])[perm]
    new_cu = np.zeros(perm.size + 1, np.int64)
    np.cumsum(lens, out=new_cu[1:])
    return calls, perm, new_cu


def adversarial_order(sizes: Sequence[int], b_min: int) -> np.ndarray:
    """A partition arrival order that stresses the aggregator (Sec. 3.2): the
    smallest partitions first, as many as keep the running total below
    B_min, then the largest partition, then the rest in their order."""
    sizes = np.asarray(sizes, np.int64)
    big = int(np.argmax(sizes))
    head, total = [], 0
    for p in np.argsort(sizes, kind="stable"):
        if p == big or sizes[p] == 0:
            continue
        if total + sizes[p] >= b_min:
            break
        head.append(int(p))
        total += int(sizes[p])
    used = set(head) | {big}
    return np.array(head + [big] + [p for p in range(sizes.size) if p not in used], np.int64)


def plan_stats(calls: List[Call], cu: np.ndarray, d: int) -> Dict:
    """Largest call and Lemma 1's data-resident size of it, M(S) = S L + 4 S d
    bytes with the text part counted as int32 token IDs."""
    texts = np.array([t1 - t0 for t0, t1, _ in calls], np.int64)
    toks = np.array([cu[t1] - cu[t0] for t0, t1, _ in calls], np.int64)
    k = int(np.argmax(texts))
    return {"calls": len(calls), "max_texts": int(texts[k]), "max_tokens": int(toks.max()),
            "mem_bytes": int(toks[k] * 4 + 4 * texts[k] * d)}


def ipc_speedup(alpha: float, n_calls_surge: int, n_parts: int) -> float:
    """Theorem 1: T_PBP / T_SURGE = (1 + a) / (1 + a F / P)."""
    return (1.0 + alpha) / (1.0 + alpha * n_calls_surge / n_parts)


def fit_call_cost(texts: np.ndarray, ms: np.ndarray) -> Tuple[float, float]:
    """Least-squares (c_call, c_enc) in ms of T = c_call + n c_enc."""
    A = np.stack([np.ones_like(texts, dtype=np.float64), texts.astype(np.float64)], axis=1)
    (c0, c1), *_ = np.linalg.lstsq(A, ms.astype(np.float64), rcond=None)
    return float(c0), float(c1)


def run_calls(torch, enc, wl, calls: List[Call], tok, out, stream, cu=None) -> Dict:
    """Encode every call in order on `stream`; per-call and total event times.
    `tok` (device) holds the texts in the layout `cu` describes (default: the
    input's own); rows go to the input's partitions."""
    d = out.shape[1]
    ptrs = np.array([out.data_ptr() + int(o) * d * 4 for o in wl.part_offsets[:-1]], np.uint64)
    sizes = np.diff(wl.part_offsets).astype(np.int64)
    cu = wl.cu_seqlens if cu is None else cu
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for k, (t0, t1, segs) in enumerate(calls):
        lcu = cu[t0:t1 + 1] - cu[t0]
        enc.encode_superbatch(t1 - t0, int(lcu[-1]), tok.data_ptr() + 4 * int(cu[t0]), lcu, segs,
                              ptrs, sizes, stream)
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    enc.check(stream)
    call_ms = np.array([evs[k].elapsed_time(evs[k + 1]) for k in range(len(calls))])
    texts = np.array([t1 - t0 for t0, t1, _ in calls])
    return {"calls": len(calls), "total_ms": float(evs[0].elapsed_time(evs[-1])),
            "call_ms": call_ms, "call_texts": texts, "first_call_ms": float(call_ms[0])}


def permuted_tokens(tokens: np.ndarray, cu: np.ndarray, perm: np.ndarray) -> np.ndarray:
    """The token IDs of texts perm[0], perm[1], ... back to back."""
    lens = cu[1:] - cu[:-1]
    starts = np.repeat(cu[:-1][perm], lens[perm])
    within = np.arange(int(lens[perm].sum())) - np.repeat(np.cumsum(lens[perm]) - lens[perm],
                                                          lens[perm])
    return tokens[starts + within]


def reorder_partitions(part_offsets: np.ndarray, cu: np.ndarray,
                       order: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """part_offsets and cu_seqlens of the same partitions arriving in `order`."""
    sizes = np.diff(part_offsets)[order]
    offs = np.zeros(order.size + 1, np.int64)
    np.cumsum(sizes, out=offs[1:])
    perm = np.concatenate([np.arange(part_offsets[p], part_offsets[p + 1]) for p in order])
    lens = (cu[1:] - cu[:-1])[perm]
    new_cu = np.zeros(perm.size + 1, np.int64)
    np.cumsum(lens, out=new_cu[1:])
    return offs, new_cu


def lemma1_table(wl, b_min: int, n_max: int, d: int) -> List[Dict]:
    """Largest SuperBatch and its M(S) (Lemma 1) under R1, R2 and FFD, for the
    input's arrival order and an adversarial one; host planning only."""
    rows = []
    n_big = int(np.diff(wl.part_offsets).max())
    for order_name in ("arrival", "adversarial"):
        if order_name == "arrival":
            offs, cu = wl.part_offsets, wl.cu_seqlens
        else:
            offs, cu = reorder_partitions(wl.part_offsets, wl.cu_seqlens,
                                          adversarial_order(np.diff(wl.part_offsets), b_min))
        for name, calls, ccu, bound in (
                ("R2", plan_surge(offs, b_min, n_max, S.SURGE_POLICY_SPLIT), cu, n_max),
                ("R1", plan_surge(offs, b_min, n_max, S.SURGE_POLICY_LITERAL), cu,
                 b_min - 1 + n_big),
                ("FFD", *plan_ffd(offs, cu, n_max)[0::2], max(n_max, n_big))):
            st = plan_stats(calls, ccu, d)
            st.update({"order": order_name, "plan": name, "bound_texts": bound,
                       "within_bound": st["max_texts"] <= bound})
            rows.append(st)
    return rows


def flops_of(shape: W.EncoderShape, lengths: np.ndarray) -> float:
    L = lengths.astype(np.float64)
    d, f = shape.d_model, shape.d_ff
    return float(shape.n_layers * np.sum(2 * L * (4 * d * d + 2 * d * f) + 4 * d * L * L))


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="bge", choices=sorted(W.WORKLOADS))
    ap.add_argument("--fsb", type=int, default=5000, help="FSB chunk size (texts)")
    ap.add_argument("--bmin", default="128,256,512,1024,2048,4096,8192,16384",
                    help="B_min values of the SURGE sweep")
    ap.add_argument("--ffd", type=int, default=5000, help="PB-PBP-LB batch capacity (texts)")
    ap.add_argument("--lemma-workload", default="minilm_heavy", choices=sorted(W.WORKLOADS),
                    help="workload of the host-only Lemma 1 table")
    ap.add_argument("--chunk-tokens", type=int, default=1 << 20)
    ap.add_argument("--markdown", default=None, help="also write a summary table here")
    args = ap.parse_args(argv)
    import torch
    assert torch.cuda.is_available(), "needs a GPU"
    torch.cuda.set_device(0)
    spec = W.WORKLOADS[args.workload]
    sh = spec.encoder
    wl = W.make_workload(spec)
    weights = W.make_weights(sh, seed=spec.seed)
    desc = S.make_desc(sh.n_layers, sh.d_model, sh.n_heads, sh.d_ff, sh.vocab_size,
                       sh.max_positions, sh.ln_eps)
    enc = S.Encoder(desc, [weights[n] for n in W.weight_names(sh.n_layers)], args.chunk_tokens)
    tok = torch.from_numpy(wl.tokens).cuda()
    out = torch.empty((wl.n_texts, sh.d_model), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    flops = flops_of(sh, wl.lengths)
    peak = 2516.6e12
    n_parts = int(np.count_nonzero(np.diff(wl.part_offsets)))

    def summary(r):
        return {"calls": r["calls"], "total_ms": r["total_ms"],
                "texts_per_s": wl.n_texts / (r["total_ms"] / 1e3),
                "mfma_util_pct": 100.0 * flops / (r["total_ms"] / 1e3) / peak,
                "first_call_ms": r["first_call_ms"], "max_call_texts": int(r["call_texts"].max())}

    # warm-up (kernels loaded, clocks up)
    run_calls(torch, enc, wl, plan_surge(wl.part_offsets, spec.b_min, spec.n_max), tok, out, stream)
    res = {"workload": args.workload, "n_texts": wl.n_texts, "n_parts": n_parts,
           "n_tokens": wl.n_tokens}
    pbp = run_calls(torch, enc, wl, plan_pbp(wl.part_offsets), tok, out, stream)
    sur = run_calls(torch, enc, wl, plan_surge(wl.part_offsets, spec.b_min, spec.n_max), tok, out,
                    stream)
    fsb = run_calls(torch, enc, wl, plan_fsb(wl.part_offsets, args.fsb), tok, out, stream)
    r1 = run_calls(torch, enc, wl, plan_surge(wl.part_offsets, spec.b_min, spec.n_max,
                                              S.SURGE_POLICY_LITERAL), tok, out, stream)
    ffd_calls, ffd_perm, ffd_cu = plan_ffd(wl.part_offsets, wl.cu_seqlens, args.ffd)
    tok_ffd = torch.from_numpy(permuted_tokens(wl.tokens, wl.cu_seqlens, ffd_perm)).cuda()
    ffd = run_calls(torch, enc, wl, ffd_calls, tok_ffd, out, stream, cu=ffd_cu)
    del tok_ffd
    c_call, c_enc = fit_call_cost(pbp["call_texts"], pbp["call_ms"])
    alpha = n_parts * c_call / (wl.n_texts * c_enc)
    pred = ipc_speedup(alpha, sur["calls"], n_parts)
    meas = pbp["total_ms"] / sur["total_ms"]
    res.update({
        "pbp": summary(pbp), "surge": summary(sur), "surge_r1": summary(r1),
        f"fsb_{args.fsb}": summary(fsb), f"ffd_{args.ffd}": summary(ffd),
        "c_call_ms": c_call, "c_enc_us_per_text": 1e3 * c_enc, "alpha": alpha,
        "n_star_texts": c_call / c_enc,
        "phi": float(np.mean(np.diff(wl.part_offsets)[np.diff(wl.part_offsets) > 0] < c_call / c_enc)),
        "speedup_predicted": pred, "speedup_measured": meas,
        "prediction_error_pct": 100.0 * (pred - meas) / meas,
        "pbp_host_gap_ms": pbp["total_ms"] - float(pbp["call_ms"].sum()),
    })
    sweep = []
    for b in [int(x) for x in args.bmin.split(",") if x]:
        r = run_calls(torch, enc, wl, plan_surge(wl.part_offsets, b, max(spec.n_max, 2 * b)), tok,
                      out, stream)
        e = summary(r)
        e.update({"b_min": b, "n_max": max(spec.n_max, 2 * b),
                  "mean_texts_per_call": wl.n_texts / r["calls"]})
        sweep.append(e)
    res["bmin_sweep"] = sweep
    enc.close()
    lspec = W.WORKLOADS[args.lemma_workload]
    res["lemma1"] = {"workload": args.lemma_workload, "b_min": lspec.b_min, "n_max": lspec.n_max,
                     "largest_partition": int(np.diff(W.make_workload(lspec).part_offsets).max()),
                     "rows": lemma1_table(W.make_workload(lspec), lspec.b_min, lspec.n_max,
                                          lspec.encoder.d_model)}
    print(json.dumps(res), flush=True)
    if args.markdown:
        with open(args.markdown, "w") as f:
            f.write(markdown(res, " ".join(["python -m paper_2605_01060_amd.callcost"] +
                                           (argv if argv is not None else sys.argv[1:]))))
    return 0


def markdown(res: Dict, command: str) -> str:
    fsb_key = [k for k in res if k.startswith("fsb_")][0]
    ffd_key = [k for k in res if k.startswith("ffd_")][0]
    lines = [f"Command: `{command}`", "",
             f"Workload `{res['workload']}`: {res['n_texts']} texts, {res['n_parts']} partitions, "
             f"{res['n_tokens']} tokens; one MI355X; per-call times from stream events.", "",
             "| plan | calls | largest call (texts) | first call ms | total ms | texts/s | "
             "MFMA util % |", "|---|---|---|---|---|---|---|"]
    for k in ("pbp", "surge", "surge_r1", fsb_key, ffd_key):
        r = res[k]
        lines.append(f"| {k} | {r['calls']} | {r['max_call_texts']} | {r['first_call_ms']:.1f} | "
                     f"{r['total_ms']:.1f} | {r['texts_per_s']:.0f} | {r['mfma_util_pct']:.1f} |")
    lines += ["", f"Fit over the PBP calls: c_call = {res['c_call_ms']:.3f} ms, "
                  f"c_enc = {res['c_enc_us_per_text']:.2f} µs/text, n* = {res['n_star_texts']:.0f} "
                  f"texts, phi = {res['phi']:.2f}, alpha = {res['alpha']:.3f}.",
              f"Theorem 1: predicted PBP/SURGE speedup {res['speedup_predicted']:.3f}, measured "
              f"{res['speedup_measured']:.3f} (error {res['prediction_error_pct']:+.1f} %).", "",
              "| B_min | n_max | calls | texts/call | texts/s | MFMA util % |",
              "|---|---|---|---|---|---|"]
    for e in res["bmin_sweep"]:
        lines.append(f"| {e['b_min']} | {e['n_max']} | {e['calls']} | "
                     f"{e['mean_texts_per_call']:.0f} | {e['texts_per_s']:.0f} | "
                     f"{e['mfma_util_pct']:.1f} |")
    lm = res["lemma1"]
    lines += ["", f"Lemma 1 on `{lm['workload']}` (host planning only): B_min = {lm['b_min']}, "
                  f"n_max (cap) = {lm['n_max']}, largest partition {lm['largest_partition']} texts; "
                  "M(S) = 4 bytes per token + 4 d bytes per text of the largest call.", "",
              "| arrival order | plan | calls | largest call (texts) | bound (texts) | M(S) MB |",
              "|---|---|---|---|---|---|"]
    for r in lm["rows"]:
        lines.append(f"| {r['order']} | {r['plan']} | {r['calls']} | {r['max_texts']} | "
                     f"{r['bound_texts']} | {r['mem_bytes'] / 1e6:.1f} |")
    return "\n".join(lines) + "\n"


if __name__ == "__main__":
    sys.exit(main())
