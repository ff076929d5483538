"""The same texts encoded under every plan of the cost-model comparison: one
call per partition (PBP, Sec. 2.2), fixed chunks across partition boundaries
(FSB, Sec. 2.2), SURGE SuperBatches under both readings of Alg. 1 (R2 split,
R1 literal) and FFD-packed whole partitions (PB-PBP-LB, Sec. 5.3).

Each plan's rows are compared with the float32 oracle at the first and last
text of every call (plus random texts), and all plans must give
bit-identical rows: a text's result does not depend on which call it rides
in (the premise of Sec. 2.2's comparison), and every row lands in its
partition's segment (outputs are NaN-filled before every run).
"""
import dataclasses

import numpy as np
import pytest

from gpu_util import assert_parity, desc_of, torch_cuda, weight_list
from oracle import encoder as E
from paper_2605_01060_amd import callcost as CC
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu


def test_plans_match_oracle_and_each_other():
    torch = torch_cuda()
    spec = dataclasses.replace(W.WORKLOADS["minilm"], n_texts=12000, n_parts=48)
    wl = W.make_workload(spec)
    sh = spec.encoder
    weights = W.make_weights(sh, seed=spec.seed)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    tok = torch.from_numpy(wl.tokens).cuda()
    stream = torch.cuda.current_stream()
    plans = {"surge_r2": CC.plan_surge(wl.part_offsets, 1000, 1500),
             "surge_r1": CC.plan_surge(wl.part_offsets, 1000, 1500, S.SURGE_POLICY_LITERAL),
             "pbp": CC.plan_pbp(wl.part_offsets),
             "fsb": CC.plan_fsb(wl.part_offsets, 777)}
    outs, edges = {}, {}
    for name, calls in plans.items():
        out = torch.full((wl.n_texts, sh.d_model), float("nan"), device="cuda")
        r = CC.run_calls(torch, enc, wl, calls, tok, out, stream)
        print(f"[plans] {name}: {r['calls']} calls, {r['total_ms']:.2f} ms", flush=True)
        assert r["calls"] == len(calls) and np.all(r["call_ms"] > 0)
        outs[name] = out.cpu().numpy()
        edges[name] = sorted({t for t0, t1, _ in calls for t in (t0, t1 - 1)})
    # PB-PBP-LB: FFD batches of whole partitions, texts re-laid out batch by batch
    calls, perm, cu = CC.plan_ffd(wl.part_offsets, wl.cu_seqlens, 2500)
    tok_ffd = torch.from_numpy(CC.permuted_tokens(wl.tokens, wl.cu_seqlens, perm)).cuda()
    out = torch.full((wl.n_texts, sh.d_model), float("nan"), device="cuda")
    r = CC.run_calls(torch, enc, wl, calls, tok_ffd, out, stream, cu=cu)
    print(f"[plans] ffd: {r['calls']} calls, {r['total_ms']:.2f} ms", flush=True)
    outs["ffd"] = out.cpu().numpy()
    edges["ffd"] = sorted({int(perm[t]) for t0, t1, _ in calls for t in (t0, t1 - 1)})
    enc.close()

    rng = np.random.default_rng(1)
    extra = rng.choice(wl.n_texts, size=16, replace=False).tolist()
    want = sorted(set(extra).union(*edges.values()))
    w32 = E.as_f32(weights)
    ref = dict(zip(want, E.encode_texts(w32, sh.n_layers, sh.n_heads, wl.tokens, wl.cu_seqlens,
                                        want, sh.ln_eps)))
    for name, got in outs.items():
        assert not np.isnan(got).any(), name
        idx = sorted(set(edges[name]) | set(extra))
        print(f"[plans] {name}: {len(idx)} rows against the oracle", flush=True)
        assert_parity(got[idx], np.stack([ref[i] for i in idx]), "minilm")
    for name in ("surge_r1", "pbp", "fsb", "ffd"):
        np.testing.assert_array_equal(outs[name], outs["surge_r2"])
