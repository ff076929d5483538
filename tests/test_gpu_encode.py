"""End-to-end parity of SuperBatch encoding through the C-ABI.

Every configuration runs the whole workload through surge_encode_all (the
call the benchmark times); the tiny one is compared on every text, the full
sized ones on a sample that covers the first and last text of SuperBatches
and the rows around every split-partition boundary.  Outputs are NaN-filled
before the call, so a row never written (or written to the wrong place)
shows up.
"""
import numpy as np
import pytest

from gpu_util import assert_parity, desc_of, torch_cuda, weight_list
from oracle import encoder as E
from oracle import plan as OP
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu

_cache = {}


def _setup(name):
    if name not in _cache:
        spec = W.WORKLOADS[name]
        wl = W.make_workload(spec)
        weights = W.make_weights(spec.encoder, seed=spec.seed)
        _cache.clear()
        _cache[name] = (spec, wl, weights)
    return _cache[name]


def _outputs(torch, wl, d):
    out = torch.full((wl.n_texts, d), float("nan"), device="cuda")
    ptrs = np.array([out.data_ptr() + int(o) * d * 4 for o in wl.part_offsets[:-1]],
                    dtype=np.uint64)
    return out, ptrs


def _encode_all(torch, enc, wl, d, b_min, n_max, policy=S.SURGE_POLICY_SPLIT):
    out, ptrs = _outputs(torch, wl, d)
    tok = torch.from_numpy(wl.tokens).cuda()
    stream = torch.cuda.current_stream()
    nsb = enc.encode_all(wl.n_texts, tok, wl.cu_seqlens, wl.part_offsets, b_min, n_max, ptrs,
                         policy=policy, stream=stream)
    enc.check(stream)
    torch.cuda.synchronize()
    return out.cpu().numpy(), nsb


def _oracle_rows(spec, weights, wl, idx):
    w = E.as_f32(weights)
    sh = spec.encoder
    return E.encode_texts(w, sh.n_layers, sh.n_heads, wl.tokens, wl.cu_seqlens, idx, sh.ln_eps)


def _sample(spec, wl, n_random, n_sb, seed=0):
    """Texts to compare: SuperBatch ends, split-partition boundaries, random."""
    sbs = OP.plan(wl.part_offsets, spec.b_min, spec.n_max, OP.R2)
    idx = {0, wl.n_texts - 1}
    for sb in sbs[:n_sb] + sbs[-2:]:
        idx.update({sb.text_begin, sb.text_end - 1})
    for sb in sbs:
        for s in sb.segments:
            if s.row_offset > 0:
                idx.update({s.first_text - 1, s.first_text})
    rng = np.random.default_rng(seed)
    idx.update(rng.choice(wl.n_texts, size=n_random, replace=False).tolist())
    return sorted(idx), sbs


def test_tiny_all_texts():
    torch = torch_cuda()
    spec, wl, weights = _setup("tiny")
    sh = spec.encoder
    print(f"[tiny] texts={wl.n_texts} tokens={wl.n_tokens}", flush=True)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    got, nsb = _encode_all(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max)
    assert nsb == 1
    assert not np.isnan(got).any()
    ref = _oracle_rows(spec, weights, wl, range(wl.n_texts))
    assert_parity(got, ref, "tiny")
    enc.close()


def test_tiny_invariant_to_composition_and_chunking():
    """A text's embedding is bit-identical whatever SuperBatch it lands in,
    whatever policy formed the SuperBatches and wherever chunks are cut."""
    torch = torch_cuda()
    spec, wl, weights = _setup("tiny")
    sh = spec.encoder
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    a, _ = _encode_all(torch, enc, wl, sh.d_model, spec.b_min, 0)
    b, nb = _encode_all(torch, enc, wl, sh.d_model, 37, 60)  # many SuperBatches, splits
    c, nc = _encode_all(torch, enc, wl, sh.d_model, 100, 0, S.SURGE_POLICY_LITERAL)
    enc.close()
    small = S.Encoder(desc_of(sh), weight_list(sh, weights), 64)  # one text per chunk or so
    d, _ = _encode_all(torch, small, wl, sh.d_model, spec.b_min, 0)
    small.close()
    assert nb > 10 and nc > 5
    assert np.array_equal(a, b)
    assert np.array_equal(a, c)
    assert np.array_equal(a, d)


def test_bge_invariant_across_tile_configurations():
    """bge shapes (d = 768): a chunk of fewer than 8192 tokens runs the
    128 x 128 GEMM tiles, a larger one the 256 x 256 tiles; the folded
    LayerNorms' row statistics are built from the same 64-feature partials
    in both, so every text's embedding is bit-identical either way."""
    import dataclasses
    torch = torch_cuda()
    spec = dataclasses.replace(W.WORKLOADS["bge"], n_texts=400, n_parts=8)
    wl = W.make_workload(spec)
    sh = spec.encoder
    weights = W.make_weights(sh, seed=spec.seed)
    assert wl.n_tokens > 2 * 8192
    big = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)  # one chunk, 256-wide tiles
    a, _ = _encode_all(torch, big, wl, sh.d_model, wl.n_texts, 0)
    b, nb = _encode_all(torch, big, wl, sh.d_model, 50, 80)  # small SuperBatches
    big.close()
    small = S.Encoder(desc_of(sh), weight_list(sh, weights), 4096)  # chunks < 8192 tokens
    c, _ = _encode_all(torch, small, wl, sh.d_model, wl.n_texts, 0)
    small.close()
    assert nb > 4
    assert not np.isnan(a).any()
    assert np.array_equal(a, b)
    assert np.array_equal(a, c)


def test_superbatch_entry_point_with_split_partition():
    """surge_encode_superbatch with a hand-made segment table: a SuperBatch
    holding the tail of one partition (row_offset > 0) and the head of the
    next, written into partitions with guard rows left untouched."""
    torch = torch_cuda()
    spec, wl, weights = _setup("tiny")
    sh = spec.encoder
    d = sh.d_model
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    texts = list(range(100, 130))  # global texts 100..129
    cu = wl.cu_seqlens[100:131] - wl.cu_seqlens[100]
    tok = torch.from_numpy(wl.tokens[wl.cu_seqlens[100]:wl.cu_seqlens[130]].copy()).cuda()
    part_sizes = np.array([50, 40], dtype=np.int64)
    outs = [torch.full((n, d), float("nan"), device="cuda") for n in part_sizes]
    ptrs = np.array([o.data_ptr() for o in outs], dtype=np.uint64)
    segs = S.segments_array([(0, 12, 0, 38), (12, 18, 1, 0)])
    enc.encode_superbatch(30, int(cu[-1]), tok, cu, segs, ptrs, part_sizes,
                          stream=torch.cuda.current_stream())
    enc.check()
    torch.cuda.synchronize()
    p0 = outs[0].cpu().numpy()
    p1 = outs[1].cpu().numpy()
    assert np.isnan(p0[:38]).all() and np.isnan(p1[18:]).all()
    ref = _oracle_rows(spec, weights, wl, texts)
    got = np.concatenate([p0[38:50], p1[:18]])
    assert_parity(got, ref, "tiny")
    enc.close()


def test_edge_cases_empty_partitions_and_extreme_lengths():
    torch = torch_cuda()
    spec = W.WORKLOADS["tiny"]
    sh = spec.encoder
    lengths = [1, 64, 2, 64, 1, 3, 64, 1, 2, 33]
    sizes = [0, 3, 0, 0, 5, 2, 0]
    wl = W.workload_from_lengths(spec, sizes, lengths, seed=4)
    weights = W.make_weights(sh, seed=1)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 128)
    got, nsb = _encode_all(torch, enc, wl, sh.d_model, 2, 3)
    assert not np.isnan(got).any()
    ref = _oracle_rows(spec, weights, wl, range(wl.n_texts))
    assert_parity(got, ref, "tiny")
    # n_texts = 0 is a no-op.
    empty = W.workload_from_lengths(spec, [0, 0], [], seed=4)
    out = torch.zeros((1, sh.d_model), device="cuda")
    enc.encode_all(0, out, empty.cu_seqlens, empty.part_offsets, 2, 3,
                   np.array([out.data_ptr(), out.data_ptr()], dtype=np.uint64))
    enc.close()


def test_invalid_arguments_write_nothing():
    torch = torch_cuda()
    spec, wl, weights = _setup("tiny")
    sh = spec.encoder
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    out, ptrs = _outputs(torch, wl, sh.d_model)
    tok = torch.from_numpy(wl.tokens).cuda()
    bad_cu = wl.cu_seqlens.copy()
    bad_cu[5] = bad_cu[4]  # a zero-length text
    with pytest.raises(S.SurgeError) as ei:
        enc.encode_all(wl.n_texts, tok, bad_cu, wl.part_offsets, 1000, 0, ptrs)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
    bad_ptrs = ptrs.copy()
    bad_ptrs[3] += 4  # misaligned output
    with pytest.raises(S.SurgeError):
        enc.encode_all(wl.n_texts, tok, wl.cu_seqlens, wl.part_offsets, 1000, 0, bad_ptrs)
    torch.cuda.synchronize()
    assert torch.isnan(out).all()
    enc.close()


def test_out_of_vocab_token_is_reported():
    torch = torch_cuda()
    spec, wl, weights = _setup("tiny")
    sh = spec.encoder
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    toks = wl.tokens.copy()
    toks[10] = sh.vocab_size + 5
    out, ptrs = _outputs(torch, wl, sh.d_model)
    enc.encode_all(wl.n_texts, torch.from_numpy(toks).cuda(), wl.cu_seqlens, wl.part_offsets,
                   1000, 0, ptrs)
    with pytest.raises(S.SurgeError) as ei:
        enc.check()
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
    enc.check()  # the flag is cleared
    enc.close()


@pytest.mark.parametrize("name,n_random,n_sb", [("minilm", 40, 8), ("bge", 24, 6),
                                                ("minilm_heavy", 24, 8), ("large", 4, 2),
                                                ("bge_s1", 8, 2)])
def test_full_workload_sampled(name, n_random, n_sb):
    torch = torch_cuda()
    spec, wl, weights = _setup(name)
    sh = spec.encoder
    print(f"[{name}] texts={wl.n_texts} tokens={wl.n_tokens}", flush=True)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 20)  # the benchmark's chunk
    got, nsb = _encode_all(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max)
    enc.close()
    idx, sbs = _sample(spec, wl, n_random, n_sb)
    assert nsb == len(sbs)
    assert not np.isnan(got).any()
    norms = np.linalg.norm(got.astype(np.float64), axis=1)
    assert np.max(np.abs(norms - 1.0)) < 1e-5
    ref = _oracle_rows(spec, weights, wl, idx)
    assert_parity(got[idx], ref, name)


def test_profile_select_times_only_the_selected_class():
    """Kernel-class selection: with every class timed and with one class
    selected, the selected class records the same launches and the others
    none; the outputs are unchanged and a mask beyond the last class is an
    argument error."""
    torch = torch_cuda()
    spec, wl, weights = _setup("tiny")
    sh = spec.encoder
    print("[profile_select] tiny workload", flush=True)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    enc.profile(True)
    ref, _ = _encode_all(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max)
    every = enc.profile_read()
    enc.profile(True, kinds=["ffn1"])
    got, _ = _encode_all(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max)
    one = enc.profile_read()
    enc.profile(False)
    assert np.array_equal(ref, got)
    assert every["ffn1"]["launches"] == sh.n_layers
    assert all(every[k]["launches"] > 0 for k in S.KERNEL_NAMES if k not in ("ln1", "ln2"))
    for k in S.KERNEL_NAMES:
        want = every[k]["launches"] if k == "ffn1" else 0
        assert one[k]["launches"] == want, k
    assert one["ffn1"]["flops"] == every["ffn1"]["flops"]
    with pytest.raises(S.SurgeError):
        S._check(S.lib().surge_profile_select(enc.handle, 1 << len(S.KERNEL_NAMES)))


@pytest.mark.parametrize("name", ["bge", "minilm", "large"])
def test_texts_at_the_position_limit(name):
    """Each encoder shape end to end with texts of the maximum length (every
    learned position; 16 key blocks of attention for bge and large) next to
    one- and two-token texts, an empty partition and a 32/33-token block
    boundary, every text against the oracle."""
    torch = torch_cuda()
    spec = W.WORKLOADS[name]
    sh = spec.encoder
    P = sh.max_positions
    lengths = [P, 1, P - 1, 2, min(300, P - 3), 33, 32, P]
    wl = W.workload_from_lengths(spec, [3, 0, 4, 1], lengths, seed=5)
    weights = W.make_weights(sh, seed=2)
    print(f"[{name} max length] lengths={lengths}", flush=True)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 12)
    got, nsb = _encode_all(torch, enc, wl, sh.d_model, 3, 0)
    enc.close()
    assert not np.isnan(got).any()
    ref = _oracle_rows(spec, weights, wl, range(wl.n_texts))
    assert_parity(got, ref, name)


@pytest.mark.parametrize("name", ["tiny", "bge"])
def test_bert_style_init_end_to_end(name):
    """BERT-style initialisation (biases 0, LayerNorm gamma 1, beta 0) end
    to end, every text against the oracle: the degenerate affine parameters
    the folded LayerNorm epilogues must also get right."""
    torch = torch_cuda()
    spec = W.WORKLOADS[name]
    sh = spec.encoder
    base = W.make_workload(spec)
    n = 160
    sizes = [40, 0, 1, 79, 40]
    wl = W.workload_from_lengths(spec, sizes, base.lengths[:n], seed=8)
    weights = W.make_weights(sh, seed=3, init="bert")
    assert not weights["layer0.b_qkv"].any() and (weights["layer0.ln1_g"] == 1).all()
    print(f"[bert init {name}] texts={wl.n_texts} tokens={wl.n_tokens}", flush=True)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    got, _ = _encode_all(torch, enc, wl, sh.d_model, 64, 100)
    enc.close()
    assert not np.isnan(got).any()
    ref = _oracle_rows(spec, weights, wl, range(wl.n_texts))
    assert_parity(got, ref, name)


def test_bf16_host_weights_give_the_same_encoder():
    """An encoder created from bf16 host arrays (a bf16 checkpoint) and one
    created from float32 arrays holding the same values produce bit-identical
    embeddings (bge shapes, whose weights are bf16-valued)."""
    torch = torch_cuda()
    import dataclasses
    spec = dataclasses.replace(W.WORKLOADS["bge"], n_texts=600, n_parts=12)
    wl = W.make_workload(spec)
    sh = spec.encoder
    weights = W.make_weights(sh, seed=spec.seed)
    f32 = weight_list(sh, weights)
    bits = []
    for a in f32:
        u = np.ascontiguousarray(a, np.float32).view(np.uint32)
        assert not (u & 0xFFFF).any()  # bf16-representable
        bits.append((u >> 16).astype(np.uint16))
    print(f"[bf16 weights] texts={wl.n_texts} tokens={wl.n_tokens}", flush=True)
    a_enc = S.Encoder(desc_of(sh), f32, 1 << 16)
    a, _ = _encode_all(torch, a_enc, wl, sh.d_model, spec.b_min, spec.n_max)
    a_enc.close()
    desc = desc_of(sh)
    desc.weight_dtype = S.SURGE_WEIGHTS_BF16
    b_enc = S.Encoder(desc, bits, 1 << 16)
    b, _ = _encode_all(torch, b_enc, wl, sh.d_model, spec.b_min, spec.n_max)
    b_enc.close()
    assert not np.isnan(a).any()
    assert np.array_equal(a, b)
    ref = _oracle_rows(spec, weights, wl, range(0, wl.n_texts, 50))
    assert_parity(b[::50], ref, "bge")


def test_calls_on_two_streams_without_host_sync():
    """Two encode_all calls of one encoder on two different streams, the
    second issued while the first may still run: the encoder orders them (its
    workspace and metadata buffers are shared), so each call's rows equal
    those of the same call made alone."""
    torch = torch_cuda()
    import dataclasses
    spec = dataclasses.replace(W.WORKLOADS["minilm"], n_texts=20000, n_parts=80)
    wl = W.make_workload(spec)
    sh = spec.encoder
    weights = W.make_weights(sh, seed=spec.seed)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    print(f"[two streams] texts={wl.n_texts} tokens={wl.n_tokens}", flush=True)
    ref, _ = _encode_all(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max)
    tok = torch.from_numpy(wl.tokens).cuda()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    torch.cuda.synchronize()
    for k, (s, b_min, n_max) in enumerate([(sa, spec.b_min, spec.n_max), (sb, 700, 900),
                                           (sa, 2500, 0), (sb, spec.b_min, spec.n_max)]):
        out, ptrs = _outputs(torch, wl, sh.d_model)
        enc.encode_all(wl.n_texts, tok, wl.cu_seqlens, wl.part_offsets, b_min, n_max, ptrs,
                       stream=s)
        outs.append(out)
    enc.check(sa)
    enc.check(sb)
    torch.cuda.synchronize()
    enc.close()
    for k, out in enumerate(outs):
        assert np.array_equal(out.cpu().numpy(), ref), f"call {k}"
