"""Streamed SuperBatch encode (host tokens in, host embeddings out) through
the C-ABI: two streams with double-buffered uploads and downloads, and the
synchronous single-stream baseline.

Both must reproduce surge_encode_all's rows bit for bit (the same kernels
run on the same SuperBatches in the same order), on a workload with enough
SuperBatches that every staging buffer is reused; the timing summary must
be consistent (Sec. 3.3's overlap ratio lies in [0, 1], the first output
arrives before the last).
"""
import dataclasses

import numpy as np
import pytest

from gpu_util import assert_parity, desc_of, torch_cuda, weight_list
from oracle import encoder as E
from oracle import plan as OP
from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

pytestmark = pytest.mark.gpu


def _workload(name, n_texts=None):
    spec = W.WORKLOADS[name]
    if n_texts is not None:
        spec = dataclasses.replace(spec, n_texts=n_texts, n_parts=max(4, n_texts // 250))
    wl = W.make_workload(spec)
    weights = W.make_weights(spec.encoder, seed=spec.seed)
    return spec, wl, weights


def _reference(torch, enc, wl, d, b_min, n_max):
    out = torch.full((wl.n_texts, d), float("nan"), device="cuda")
    ptrs = np.array([out.data_ptr() + int(o) * d * 4 for o in wl.part_offsets[:-1]],
                    dtype=np.uint64)
    tok = torch.from_numpy(wl.tokens).cuda()
    stream = torch.cuda.current_stream()
    nsb = enc.encode_all(wl.n_texts, tok, wl.cu_seqlens, wl.part_offsets, b_min, n_max, ptrs,
                         stream=stream)
    enc.check(stream)
    torch.cuda.synchronize()
    return out.cpu().numpy(), nsb


def _streamed(torch, enc, wl, d, b_min, n_max, overlap):
    h_tok = torch.from_numpy(wl.tokens).pin_memory()
    h_out = torch.full((wl.n_texts, d), float("nan")).pin_memory()
    cs = torch.cuda.Stream()
    xs = torch.cuda.Stream()
    nsb = len(OP.plan(wl.part_offsets, b_min, n_max, OP.R2))
    times = np.zeros((nsb, 3), np.float64)
    st = enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets, b_min, n_max,
                                 h_out, overlap=overlap, compute_stream=cs, copy_stream=xs,
                                 sb_times=times)
    return h_out.numpy().copy(), st, times


@pytest.mark.parametrize("overlap", [1, 0, 2])
def test_streamed_matches_encode_all(overlap):
    torch = torch_cuda()
    spec, wl, weights = _workload("minilm", n_texts=12000)
    sh = spec.encoder
    b_min, n_max = 1000, 1500  # ~10 SuperBatches: both staging buffers reused
    print(f"[stream overlap={overlap}] texts={wl.n_texts} tokens={wl.n_tokens}", flush=True)
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    ref, nsb = _reference(torch, enc, wl, sh.d_model, b_min, n_max)
    got, st, times = _streamed(torch, enc, wl, sh.d_model, b_min, n_max, overlap)
    print(f"[stream overlap={overlap}] {st}", flush=True)
    assert nsb >= 6
    assert st["n_superbatches"] == nsb
    np.testing.assert_array_equal(got, ref)
    assert st["total_ms"] > 0 and 0 < st["ttfo_ms"] <= st["total_ms"]
    assert 0.0 <= st["rho"] <= 1.0 and 0.0 <= st["rho_measured"] <= 1.0
    assert np.all(times[:, :2] > 0)
    if overlap == 2:  # zero copy: no download step
        assert np.all(times[:, 2] == 0) and st["d2h_ms"] == 0
    else:
        assert np.all(times[:, 2] > 0)
    # Lemma 1 (Sec. 4.3): the staging holds two SuperBatches' data-resident
    # state, M(S) = S L + 4 S d with the text part as int32 token IDs, for the
    # plan's largest SuperBatch (the embeddings only when they are downloaded)
    sbs = OP.plan(wl.part_offsets, b_min, n_max, OP.R2)
    max_txt = max(sb.n_texts for sb in sbs)
    max_tok = max(int(wl.cu_seqlens[sb.text_end] - wl.cu_seqlens[sb.text_begin]) for sb in sbs)
    assert (st["max_sb_texts"], st["max_sb_tokens"]) == (max_txt, max_tok)
    want = 2 * OP.device_superbatch_memory(0 if overlap == 2 else max_txt, max_tok, sh.d_model)
    assert st["staging_bytes"] == want
    assert max_txt <= OP.largest_superbatch_bound(b_min, int(np.diff(wl.part_offsets).max()),
                                                  n_max, OP.R2)
    assert st["enc_ms"] == pytest.approx(times[:, 1].sum(), rel=1e-6)
    if overlap == 0:
        # one stream: the phases add up
        assert st["total_ms"] >= 0.99 * (st["enc_ms"] + st["h2d_ms"] + st["d2h_ms"])
    # a sample against the oracle, so the streamed path is pinned on its own
    idx = [0, 1, wl.n_texts // 2, wl.n_texts - 1]
    w = E.as_f32(weights)
    oref = E.encode_texts(w, sh.n_layers, sh.n_heads, wl.tokens, wl.cu_seqlens, idx, sh.ln_eps)
    assert_parity(got[idx], oref, "minilm")


def test_streamed_tiny_single_superbatch():
    torch = torch_cuda()
    spec, wl, weights = _workload("tiny")
    sh = spec.encoder
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    ref, nsb = _reference(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max)
    got, st, _ = _streamed(torch, enc, wl, sh.d_model, spec.b_min, spec.n_max, 1)
    assert nsb == 1 and st["n_superbatches"] == 1
    np.testing.assert_array_equal(got, ref)


def test_streamed_invalid_arguments():
    torch = torch_cuda()
    spec, wl, weights = _workload("tiny")
    sh = spec.encoder
    enc = S.Encoder(desc_of(sh), weight_list(sh, weights), 1 << 16)
    h_tok = torch.from_numpy(wl.tokens).pin_memory()
    h_out = torch.zeros((wl.n_texts, sh.d_model)).pin_memory()
    cs = torch.cuda.Stream()
    with pytest.raises(S.SurgeError) as ei:  # overlap needs two streams
        enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                                spec.n_max, h_out, overlap=1, compute_stream=cs, copy_stream=cs)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
    with pytest.raises(S.SurgeError) as ei:  # no output buffer
        enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                                spec.n_max, None, overlap=0, compute_stream=cs)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
    bad = wl.part_offsets.copy()
    bad[-1] += 1
    with pytest.raises(S.SurgeError):
        enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, bad, spec.b_min, spec.n_max,
                                h_out, overlap=0, compute_stream=cs)
    # zero copy needs pinned (device-mapped) output memory: pageable memory
    # is refused before anything runs
    pageable = np.zeros((wl.n_texts, sh.d_model), np.float32)
    with pytest.raises(S.SurgeError) as ei:
        enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                                spec.n_max, pageable, overlap=2, compute_stream=cs)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
    assert np.all(pageable == 0)
    with pytest.raises(S.SurgeError) as ei:  # no such mode
        enc.encode_all_streamed(wl.n_texts, h_tok, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                                spec.n_max, h_out, overlap=3, compute_stream=cs)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
    # an out-of-vocabulary token is reported after the run
    tok = wl.tokens.copy()
    tok[5] = sh.vocab_size + 7
    h_bad = torch.from_numpy(tok).pin_memory()
    with pytest.raises(S.SurgeError) as ei:
        enc.encode_all_streamed(wl.n_texts, h_bad, wl.cu_seqlens, wl.part_offsets, spec.b_min,
                                spec.n_max, h_out, overlap=0, compute_stream=cs)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT
