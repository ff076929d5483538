"""Every row at full scale: the 1M-text heavy-tailed layout (4,000
partitions, log-normal sigma 2.5, the largest split across SuperBatches by
the n_max cap, Sec. 6) with an identity payload.

The layout, the partition sizes and the length distribution are those of the
minilm_heavy workload; the texts themselves are drawn, with replacement,
from a pool of 384 distinct texts (the workload's first 384).  A text's
embedding is a function of its own tokens only, so every output row must be
bit-identical to the row of the first text that carries the same pool
entry: a row written to the wrong place, twice, or not at all breaks that,
on any of the 10^6 rows.  The pool entries themselves are checked against
the float32 oracle, and the SURGE (split), one-call-per-partition and
fixed-chunk plans must agree on every row bit for bit.
"""
import numpy as np
import pytest

from gpu_util import assert_parity, desc_of, torch_cuda, weight_list
from oracle import encoder as E
from oracle import plan as OP
from paper_2605_01060_amd import callcost as CC
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu

N_POOL = 384


def _pooled_workload(spec, seed=2024):
    """The workload's partition layout with texts drawn from a pool of its
    first N_POOL texts; returns (workload, pool id of every text)."""
    base = W.make_workload(spec)
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, N_POOL, size=base.n_texts)
    ids[:N_POOL] = np.arange(N_POOL)  # every pool entry occurs
    rng.shuffle(ids)
    pool_len = base.lengths[:N_POOL].astype(np.int64)
    pool_cu = base.cu_seqlens[:N_POOL + 1].astype(np.int64)
    lengths = pool_len[ids]
    cu = np.zeros(base.n_texts + 1, np.int64)
    np.cumsum(lengths, out=cu[1:])
    text_of = np.repeat(np.arange(base.n_texts), lengths)
    src = pool_cu[ids][text_of] + (np.arange(int(cu[-1])) - cu[text_of])
    tokens = base.tokens[src].astype(np.int32)
    wl = W.Workload(spec, base.part_sizes, base.part_offsets, lengths, cu, tokens)
    return wl, ids


def test_heavy_layout_every_row():
    torch = torch_cuda()
    spec = W.WORKLOADS["minilm_heavy"]
    sh = spec.encoder
    d = sh.d_model
    wl, ids = _pooled_workload(spec)
    sbs = OP.plan(wl.part_offsets, spec.b_min, spec.n_max, OP.R2)
    splits = [s for sb in sbs for s in sb.segments if s.row_offset > 0]
    print(f"[heavy every row] texts={wl.n_texts} tokens={wl.n_tokens} superbatches={len(sbs)} "
          f"split pieces={len(splits)}", flush=True)
    assert splits, "the layout must exercise the oversized-partition split"
    weights = W.make_weights(sh, seed=spec.seed)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 20)
    tok = torch.from_numpy(wl.tokens).cuda()
    stream = torch.cuda.current_stream()
    ptr = lambda o: np.array([o.data_ptr() + int(p) * d * 4 for p in wl.part_offsets[:-1]],
                             np.uint64)

    out = torch.full((wl.n_texts, d), float("nan"), device="cuda")
    nsb = enc.encode_all(wl.n_texts, tok, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                         spec.n_max, ptr(out), stream=stream)
    enc.check(stream)
    assert nsb == len(sbs)
    assert not torch.isnan(out).any().item()

    # identity payload: every row equals the first row of its pool entry
    uniq, first = np.unique(ids, return_index=True)  # first text of each pool entry
    assert np.array_equal(uniq, np.arange(N_POOL))
    rep = torch.from_numpy(first[ids]).cuda()
    same = (out == out[rep]).all(dim=1)
    bad = torch.nonzero(~same).flatten()[:10].cpu().numpy()
    assert bad.size == 0, f"rows {bad.tolist()} differ from their pool entry"

    # the pool entries against the oracle, including the rows on each side
    # of every split boundary
    w32 = E.as_f32(weights)
    got = out[torch.from_numpy(first).cuda()].cpu().numpy()
    ref = E.encode_texts(w32, sh.n_layers, sh.n_heads, wl.tokens, wl.cu_seqlens, first, sh.ln_eps)
    assert_parity(got, ref, "minilm_heavy")
    for s in splits:
        for i in (s.first_text - 1, s.first_text):
            np.testing.assert_array_equal(out[i].cpu().numpy(), got[ids[i]])

    # every row bit for bit under one call per partition and fixed chunks
    for name, calls in (("pbp", CC.plan_pbp(wl.part_offsets)),
                        ("fsb", CC.plan_fsb(wl.part_offsets, 5000))):
        other = torch.full((wl.n_texts, d), float("nan"), device="cuda")
        r = CC.run_calls(torch, enc, wl, calls, tok, other, stream)
        print(f"[heavy every row] {name}: {r['calls']} calls, {r['total_ms']:.0f} ms", flush=True)
        assert torch.equal(other, out), name
        del other
    enc.close()
