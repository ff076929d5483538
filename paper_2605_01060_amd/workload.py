"""Seeded synthetic inputs for SuperBatch encoding.

This module only draws random numbers: partition sizes, text lengths, token
IDs and encoder weights.  It holds none of the encoder's or the planner's
arithmetic, so both the HIP path and the CPU oracle can be fed from it
without sharing any computation.

The paper's dataset is synthetic and not shipped (Sec. 5.1, "Dataset": 10M
texts over 4,000 partitions, log-normal partition sizes with sigma = 1.72,
short product-title texts).  The configurations below stand in for it with
the same structure: log-normal partition sizes rescaled to N, short texts
with a log-normal (or uniform) token-length mix, BERT-style CLS/SEP ends.

Recipe (one base seed per workload):
  * ``np.random.SeedSequence(seed).spawn(4)`` gives four independent streams
    [sizes, lengths, tokens, weights].
  * Partition sizes: z ~ N(0,1)^P, raw = exp(sigma z), x = raw / sum(raw) *
    (N - P), n_p = 1 + floor(x_p); the N - sum(n_p) leftover units go to the
    largest fractional parts (ties broken by lower index).  Arrival order is
    draw order.
  * Lengths (tokens, CLS and SEP included): uniform integers in [lo, hi], or
    clip(rint(exp(ln(median) + 0.5 z)), lo, hi).
  * Tokens: position 0 is CLS (101), position L-1 is SEP (102), the rest
    uniform in [1000, 30521].
  * Weights: drawn in float32 in a fixed order (see ``make_weights``); every
    matrix, embedding table, bias and LayerNorm beta ~ N(0, 0.02), every
    LayerNorm gamma = 1 + N(0, 0.02).  Configurations with bf16 weights are
    rounded to the nearest bf16 value (ties to even) and kept as float32
    arrays holding exactly those values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

CLS_ID = 101
SEP_ID = 102
TOKEN_LO = 1000
TOKEN_HI = 30521  # inclusive


@dataclasses.dataclass(frozen=True)
class EncoderShape:
    """Shape of a post-LN BERT-style encoder."""

    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    vocab_size: int
    max_positions: int
    weight_dtype: str  # "f32" or "bf16"
    ln_eps: float = 1e-12

    @property
    def d_head(self) -> int:
        return self.d_model // self.n_heads


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    """A synthetic SuperBatch-encoding workload."""

    name: str
    encoder: EncoderShape
    n_texts: int
    n_parts: int
    part_sigma: float
    length_kind: str  # "uniform" or "lognormal"
    length_lo: int
    length_hi: int
    length_median: float  # lognormal only
    b_min: int
    n_max: int  # 0 = no cap
    seed: int = 0
    length_sigma: float = 0.5


TINY = EncoderShape(2, 128, 2, 512, 30522, 64, "f32")
MINILM = EncoderShape(6, 384, 12, 1536, 30522, 128, "bf16")
BGE = EncoderShape(12, 768, 12, 3072, 30522, 512, "bf16")
LARGE = EncoderShape(24, 1024, 16, 4096, 30522, 512, "bf16")

WORKLOADS: Dict[str, WorkloadSpec] = {
    # Tiny encoder, 1,000 texts over 20 partitions, one SuperBatch.
    "tiny": WorkloadSpec("tiny", TINY, 1_000, 20, 1.72, "uniform", 8, 64, 0.0,
                         1_000, 0),
    # MiniLM-L6-shaped encoder, 100k texts over 400 partitions.
    "minilm": WorkloadSpec("minilm", MINILM, 100_000, 400, 1.72, "lognormal",
                           4, 128, 32.0, 4_096, 20_000),
    # bge-base-shaped encoder, 200k texts over 800 partitions, sigma 1.72
    # (the headline measurement) and sigma 1.0.
    "bge": WorkloadSpec("bge", BGE, 200_000, 800, 1.72, "lognormal", 4, 256,
                        48.0, 4_096, 20_000),
    "bge_s1": WorkloadSpec("bge_s1", BGE, 200_000, 800, 1.0, "lognormal", 4,
                           256, 48.0, 4_096, 20_000),
    # MiniLM-shaped encoder on a heavy-tailed layout: 1M texts over 4,000
    # partitions, sigma 2.5.  At seed 0 the largest partition holds 512,640
    # texts, well above the 50,000-text cap, so partition splitting is
    # exercised.
    "minilm_heavy": WorkloadSpec("minilm_heavy", MINILM, 1_000_000, 4_000,
                                 2.5, "lognormal", 4, 128, 32.0, 8_192,
                                 50_000),
    # ~335M-parameter encoder, 100k texts over 400 partitions.
    "large": WorkloadSpec("large", LARGE, 100_000, 400, 1.72, "lognormal", 8,
                          512, 96.0, 2_048, 10_000),
}


@dataclasses.dataclass
class Workload:
    spec: WorkloadSpec
    part_sizes: np.ndarray    # int64 [P]
    part_offsets: np.ndarray  # int64 [P+1], CSR
    lengths: np.ndarray       # int64 [N]
    cu_seqlens: np.ndarray    # int64 [N+1]
    tokens: np.ndarray        # int32 [T]

    @property
    def n_texts(self) -> int:
        return int(self.lengths.shape[0])

    @property
    def n_tokens(self) -> int:
        return int(self.tokens.shape[0])

    def text_tokens(self, i: int) -> np.ndarray:
        return self.tokens[self.cu_seqlens[i]:self.cu_seqlens[i + 1]]


def _streams(seed: int) -> List[np.random.Generator]:
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(4)]


def partition_sizes(rng: np.random.Generator, n_texts: int, n_parts: int,
                    sigma: float) -> np.ndarray:
    """Log-normal partition sizes rescaled to sum to ``n_texts``, each >= 1."""
    if n_parts <= 0:
        raise ValueError("n_parts must be positive")
    if n_texts < n_parts:
        raise ValueError("need at least one text per partition")
    z = rng.standard_normal(n_parts)
    raw = np.exp(sigma * z)
    x = raw / raw.sum() * (n_texts - n_parts)
    base = np.floor(x)
    sizes = 1 + base.astype(np.int64)
    rem = n_texts - int(sizes.sum())
    frac = x - base
    order = np.lexsort((np.arange(n_parts), -frac))
    sizes[order[:rem]] += 1
    return sizes


def text_lengths(rng: np.random.Generator, spec: WorkloadSpec, n: int) -> np.ndarray:
    if spec.length_kind == "uniform":
        return rng.integers(spec.length_lo, spec.length_hi, size=n,
                            endpoint=True).astype(np.int64)
    if spec.length_kind == "lognormal":
        z = rng.standard_normal(n)
        raw = np.rint(np.exp(np.log(spec.length_median) + spec.length_sigma * z))
        return np.clip(raw, spec.length_lo, spec.length_hi).astype(np.int64)
    raise ValueError(f"unknown length kind {spec.length_kind!r}")


def token_ids(rng: np.random.Generator, cu_seqlens: np.ndarray) -> np.ndarray:
    n_tok = int(cu_seqlens[-1])
    toks = rng.integers(TOKEN_LO, TOKEN_HI, size=n_tok, endpoint=True).astype(np.int32)
    starts = cu_seqlens[:-1]
    ends = cu_seqlens[1:]
    nonempty = ends > starts
    toks[starts[nonempty]] = CLS_ID
    toks[ends[nonempty] - 1] = SEP_ID
    return toks


def make_workload(spec: WorkloadSpec, seed: Optional[int] = None) -> Workload:
    s_sizes, s_len, s_tok, _ = _streams(spec.seed if seed is None else seed)
    sizes = partition_sizes(s_sizes, spec.n_texts, spec.n_parts, spec.part_sigma)
    offsets = np.zeros(spec.n_parts + 1, dtype=np.int64)
    np.cumsum(sizes, out=offsets[1:])
    lengths = text_lengths(s_len, spec, spec.n_texts)
    cu = np.zeros(spec.n_texts + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    toks = token_ids(s_tok, cu)
    return Workload(spec, sizes, offsets, lengths, cu, toks)


def workload_from_lengths(spec: WorkloadSpec, part_sizes, lengths,
                          seed: int = 0) -> Workload:
    """A workload with caller-chosen partition sizes and text lengths.

    Tokens are drawn from the token stream of ``seed``.  Used for edge cases
    (empty partitions, single-token texts, maximum lengths).
    """
    sizes = np.asarray(part_sizes, dtype=np.int64)
    lengths = np.asarray(lengths, dtype=np.int64)
    if int(sizes.sum()) != lengths.shape[0]:
        raise ValueError("partition sizes must sum to the number of texts")
    offsets = np.zeros(sizes.shape[0] + 1, dtype=np.int64)
    np.cumsum(sizes, out=offsets[1:])
    cu = np.zeros(lengths.shape[0] + 1, dtype=np.int64)
    np.cumsum(lengths, out=cu[1:])
    _, _, s_tok, _ = _streams(seed)
    toks = token_ids(s_tok, cu)
    return Workload(spec, sizes, offsets, lengths, cu, toks)


# ---------------------------------------------------------------------------
# Weights
# ---------------------------------------------------------------------------

LAYER_TENSORS = ("w_qkv", "b_qkv", "w_o", "b_o", "ln1_g", "ln1_b",
                 "w_1", "b_1", "w_2", "b_2", "ln2_g", "ln2_b")


def weight_names(n_layers: int) -> List[str]:
    """The fixed tensor order used by the C-ABI and by the oracle."""
    names = ["word_emb", "pos_emb", "ln_e_g", "ln_e_b"]
    for l in range(n_layers):
        names += [f"layer{l}.{t}" for t in LAYER_TENSORS]
    return names


def weight_shapes(shape: EncoderShape) -> List[Tuple[str, Tuple[int, ...]]]:
    d, f = shape.d_model, shape.d_ff
    per_layer = {
        "w_qkv": (d, 3 * d), "b_qkv": (3 * d,), "w_o": (d, d), "b_o": (d,),
        "ln1_g": (d,), "ln1_b": (d,), "w_1": (d, f), "b_1": (f,),
        "w_2": (f, d), "b_2": (d,), "ln2_g": (d,), "ln2_b": (d,),
    }
    out = [("word_emb", (shape.vocab_size, d)), ("pos_emb", (shape.max_positions, d)),
           ("ln_e_g", (d,)), ("ln_e_b", (d,))]
    for l in range(shape.n_layers):
        out += [(f"layer{l}.{t}", per_layer[t]) for t in LAYER_TENSORS]
    return out


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value (ties to even) of each float32, as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    out = r.astype(np.uint32).view(np.float32).copy()
    nan = np.isnan(x)
    if nan.any():
        out[nan] = np.float32("nan")
    return out


def make_weights(shape: EncoderShape, seed: int = 0, init: str = "random",
                 stream_seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Encoder weights in the fixed order of ``weight_names``.

    Layout: matrices are [in, out] row-major (y = x W + b); ``w_qkv`` holds
    the Q, K and V projections as three column blocks of width d, and head h
    uses columns [h*d_head, (h+1)*d_head) of each block.

    ``init="random"`` draws every tensor as described in the module docstring;
    ``init="bert"`` draws matrices and tables the same way but sets biases
    and beta to 0 and gamma to 1.
    """
    if stream_seed is None:
        rng = _streams(seed)[3]
    else:
        rng = np.random.default_rng(stream_seed)
    out: Dict[str, np.ndarray] = {}
    for name, shp in weight_shapes(shape):
        kind = name.split(".")[-1]
        w = rng.standard_normal(shp, dtype=np.float32) * np.float32(0.02)
        if kind.endswith("_g"):
            w = (np.float32(1.0) + w) if init == "random" else np.ones(shp, np.float32)
        elif init == "bert" and (kind.startswith("b_") or kind.endswith("_b")):
            w = np.zeros(shp, np.float32)
        if shape.weight_dtype == "bf16":
            w = round_to_bf16(w)
        out[name] = np.ascontiguousarray(w, dtype=np.float32)
    return out


def workload_stats(w: Workload) -> Dict[str, float]:
    L = w.lengths.astype(np.float64)
    return {
        "n_texts": w.n_texts, "n_parts": int(w.part_sizes.shape[0]),
        "n_tokens": w.n_tokens, "mean_len": float(L.mean()),
        "mean_len_sq": float((L * L).mean()), "max_len": int(L.max()),
        "largest_partition": int(w.part_sizes.max()),
    }
