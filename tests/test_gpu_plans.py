"""The same texts encoded under the three plans of the cost-model
comparison (one call per partition, fixed chunks across partition
boundaries, SURGE SuperBatches, FFD-packed whole partitions) give
bit-identical rows: a text's result
does not depend on which call it rides in (the premise of Sec. 2.2's
comparison), and every row lands in its partition's segment.
"""
import dataclasses

import numpy as np
import pytest

from gpu_util import desc_of, torch_cuda, weight_list
from paper_2605_01060_amd import callcost as CC
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu


def test_plans_bit_identical():
    torch = torch_cuda()
    spec = dataclasses.replace(W.WORKLOADS["minilm"], n_texts=12000, n_parts=48)
    wl = W.make_workload(spec)
    sh = spec.encoder
    weights = W.make_weights(sh, seed=spec.seed)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    tok = torch.from_numpy(wl.tokens).cuda()
    stream = torch.cuda.current_stream()
    outs = {}
    plans = {"surge": CC.plan_surge(wl.part_offsets, 1000, 1500),
             "pbp": CC.plan_pbp(wl.part_offsets),
             "fsb": CC.plan_fsb(wl.part_offsets, 777)}
    for name, calls in plans.items():
        out = torch.full((wl.n_texts, sh.d_model), float("nan"), device="cuda")
        r = CC.run_calls(torch, enc, wl, calls, tok, out, stream)
        print(f"[plans] {name}: {r['calls']} calls, {r['total_ms']:.2f} ms", flush=True)
        assert r["calls"] == len(calls) and np.all(r["call_ms"] > 0)
        outs[name] = out.cpu().numpy()
    # PB-PBP-LB: FFD batches of whole partitions, texts re-laid out batch by batch
    calls, perm, cu = CC.plan_ffd(wl.part_offsets, wl.cu_seqlens, 2500)
    tok_ffd = torch.from_numpy(CC.permuted_tokens(wl.tokens, wl.cu_seqlens, perm)).cuda()
    out = torch.full((wl.n_texts, sh.d_model), float("nan"), device="cuda")
    r = CC.run_calls(torch, enc, wl, calls, tok_ffd, out, stream, cu=cu)
    print(f"[plans] ffd: {r['calls']} calls, {r['total_ms']:.2f} ms", flush=True)
    outs["ffd"] = out.cpu().numpy()
    assert not np.isnan(outs["surge"]).any()
    for name in ("pbp", "fsb", "ffd"):
        np.testing.assert_array_equal(outs[name], outs["surge"])
    enc.close()
