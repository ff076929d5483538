"""Seeded input generators: shapes, ranges and determinism."""
import numpy as np
import pytest

from paper_2605_01060_amd import workload as W


@pytest.mark.parametrize("name", ["tiny", "minilm", "bge", "bge_s1", "large"])
def test_workload_structure(name):
    spec = W.WORKLOADS[name]
    wl = W.make_workload(spec)
    assert wl.part_sizes.sum() == spec.n_texts and wl.part_sizes.min() >= 1
    assert wl.part_offsets[0] == 0 and wl.part_offsets[-1] == spec.n_texts
    assert wl.lengths.min() >= spec.length_lo and wl.lengths.max() <= spec.length_hi
    assert wl.lengths.max() <= spec.encoder.max_positions
    assert wl.cu_seqlens[-1] == wl.n_tokens
    starts, ends = wl.cu_seqlens[:-1], wl.cu_seqlens[1:]
    assert np.all(wl.tokens[starts] == W.CLS_ID) and np.all(wl.tokens[ends - 1] == W.SEP_ID)
    inner = np.ones(wl.n_tokens, bool)
    inner[starts] = False
    inner[ends - 1] = False
    assert wl.tokens[inner].min() >= W.TOKEN_LO and wl.tokens[inner].max() <= W.TOKEN_HI
    again = W.make_workload(spec)
    assert np.array_equal(again.tokens, wl.tokens)
    assert np.array_equal(again.part_sizes, wl.part_sizes)


def test_heavy_layout_exercises_the_split():
    spec = W.WORKLOADS["minilm_heavy"]
    rng = W._streams(spec.seed)[0]
    sizes = W.partition_sizes(rng, spec.n_texts, spec.n_parts, spec.part_sigma)
    assert sizes.max() > spec.n_max
    assert np.mean(sizes <= 5) > 0.25


def test_largest_remainder_rounding():
    rng = np.random.default_rng(0)
    for _ in range(50):
        n_parts = int(rng.integers(1, 50))
        n = n_parts + int(rng.integers(0, 1000))
        s = W.partition_sizes(rng, n, n_parts, 1.5)
        assert s.sum() == n and s.min() >= 1


def test_round_to_bf16():
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -9,
                  -2.5, 3.0e38, np.float32(1.00390625)], dtype=np.float32)
    r = W.round_to_bf16(x)
    # ties to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> 1
    assert r[0] == 1.0 and r[1] == 1.0 and r[2] == 1.0 + 2.0 ** -6
    assert r[3] == 1.0 and r[4] == -2.5
    assert np.all((r.view(np.uint32) & 0xFFFF) == 0)
    assert np.isnan(W.round_to_bf16(np.array([np.nan], np.float32)))[0]


def test_weights_order_and_dtype():
    shape = W.EncoderShape(2, 32, 2, 64, 100, 16, "bf16")
    w = W.make_weights(shape, seed=1)
    assert list(w) == W.weight_names(2)
    for k, v in w.items():
        assert v.dtype == np.float32
        assert np.all((v.view(np.uint32) & 0xFFFF) == 0), k
    assert abs(w["layer0.ln1_g"].mean() - 1.0) < 0.05
    wb = W.make_weights(shape, seed=1, init="bert")
    assert np.all(wb["layer1.b_qkv"] == 0) and np.all(wb["ln_e_g"] == 1)
