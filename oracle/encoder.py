"""Oracle: the per-text encoder forward, pooling, normalisation and placement.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Precision.  Every function computes in the floating-point type of the
weights it is given: ``as_dtype(weights, np.float32)`` gives the oracle the
GPU path is held to (plain float32 NumPy, BLAS sgemm for the products,
``scipy.special.erf`` for GELU); ``as_dtype(weights, np.float64)`` gives its
float64 twin, which pins the float32 results (they agree to cosine
>= 1 - 1e-9 and max-abs <= 1e-5 per component) and is the form compared
with the library encoder and the brute-force references.

What is computed, and where it comes from:

* Problem statement (Sec. 2.2, "Baseline Approaches"): partitions
  (k_i, T_i) with n_i texts, sum n_i = N; the output maps every partition to
  an embedding matrix E_i of shape [n_i, d].  Alg. 1's Flush encodes the
  concatenation of the buffered partitions in one call and slices the result
  back per partition, so packing only changes where and when a text is
  encoded, never its embedding.  The oracle therefore encodes every text on
  its own.
* Sec. 5.1 ("Model"): the encoder yields L2-normalised sentence embeddings.
  The paper treats the encoder as a black box; this build fixes a post-LN
  BERT-style encoder with masked mean pooling.  Readings of what the paper
  leaves open:
    - pooling is the mean over all L tokens of the text, CLS and SEP
      included (the text's own tokens are the mask; there is no padding);
    - GELU is the exact erf form, 0.5 z (1 + erf(z / sqrt 2));
    - every LayerNorm uses biased variance and eps = 1e-12; the L2 step
      divides by max(||e||, 1e-12);
    - post-LN: x <- LN(x + sublayer(x)) for attention and for the FFN;
    - no token-type embeddings (a constant type row folds into W_pos);
    - positions restart at 0 for every text;
    - attention is bidirectional within the text only, scale 1/sqrt(d_head).

Weight layout (shared convention with the library boundary, not code):
matrices are [in, out] (y = x W + b); ``w_qkv`` holds Q | K | V as column
blocks of width d, head h owns columns [h*dh, (h+1)*dh) in each block.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np
from scipy.special import erf

L2_EPS = 1e-12


def as_dtype(weights: Dict[str, np.ndarray], dtype) -> Dict[str, np.ndarray]:
    """The weights as arrays of ``dtype`` (np.float32: the oracle; np.float64:
    its twin).  The oracle's arithmetic then runs in that type: every scalar
    it mixes in is a Python float, which never widens an array."""
    return {k: np.asarray(v, dtype=dtype) for k, v in weights.items()}


def as_f32(weights: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    return as_dtype(weights, np.float32)


def as_f64(weights: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    return as_dtype(weights, np.float64)


def layer_norm(x: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float) -> np.ndarray:
    """LN(v) = gamma * (v - mean) / sqrt(var + eps) + beta, per row, biased var."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return gamma * (x - mu) / np.sqrt(var + eps) + beta


def gelu(z: np.ndarray) -> np.ndarray:
    """Exact GELU: z * Phi(z) = 0.5 z (1 + erf(z / sqrt 2))."""
    return 0.5 * z * (1.0 + erf(z / math.sqrt(2.0)))


def linear(x: np.ndarray, w: np.ndarray, b: np.ndarray) -> np.ndarray:
    """y = x W + b with W stored [in, out]."""
    return x @ w + b


def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax: subtract the row max, exponentiate, divide by the sum."""
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    return p / p.sum(axis=-1, keepdims=True)


def self_attention(qkv: np.ndarray, n_heads: int) -> np.ndarray:
    """Multi-head attention of one text.

    ``qkv`` is [L, 3d] (the text's rows of x W_qkv + b_qkv).  For each head h,
    A_h = softmax(Q_h K_h^T / sqrt(dh)) V_h over the text's own L keys; the
    heads are concatenated back to [L, d] in head order.
    """
    L, three_d = qkv.shape
    d = three_d // 3
    dh = d // n_heads
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    out = np.empty((L, d), dtype=qkv.dtype)
    for h in range(n_heads):
        cols = slice(h * dh, (h + 1) * dh)
        s = q[:, cols] @ k[:, cols].T / math.sqrt(dh)
        out[:, cols] = softmax_rows(s) @ v[:, cols]
    return out


def embed(w: Dict[str, np.ndarray], ids: np.ndarray, eps: float) -> np.ndarray:
    """x_t = LN_e(W_word[id_t] + W_pos[t]), positions counted from the text start."""
    L = ids.shape[0]
    x = w["word_emb"][ids] + w["pos_emb"][:L]
    return layer_norm(x, w["ln_e_g"], w["ln_e_b"], eps)


def encoder_layer(w: Dict[str, np.ndarray], l: int, x: np.ndarray, n_heads: int,
                  eps: float) -> np.ndarray:
    """One post-LN layer: attention block then FFN block, each LN(x + f(x))."""
    p = f"layer{l}."
    qkv = linear(x, w[p + "w_qkv"], w[p + "b_qkv"])
    a = self_attention(qkv, n_heads)
    x = layer_norm(x + linear(a, w[p + "w_o"], w[p + "b_o"]),
                   w[p + "ln1_g"], w[p + "ln1_b"], eps)
    hdn = gelu(linear(x, w[p + "w_1"], w[p + "b_1"]))
    x = layer_norm(x + linear(hdn, w[p + "w_2"], w[p + "b_2"]),
                   w[p + "ln2_g"], w[p + "ln2_b"], eps)
    return x


def hidden_states(w: Dict[str, np.ndarray], n_layers: int, n_heads: int,
                  ids: np.ndarray, eps: float = 1e-12) -> np.ndarray:
    """Final-layer token states [L, d] of one text."""
    x = embed(w, ids, eps)
    for l in range(n_layers):
        x = encoder_layer(w, l, x, n_heads, eps)
    return x


def mean_pool_l2(x: np.ndarray) -> np.ndarray:
    """e = (1/L) sum_t x_t; return e / max(||e||_2, 1e-12)."""
    e = x.mean(axis=0)
    return e / max(float(np.linalg.norm(e)), L2_EPS)


def encode_text(w: Dict[str, np.ndarray], n_layers: int, n_heads: int,
                ids: np.ndarray, eps: float = 1e-12) -> np.ndarray:
    """The embedding of one text ([d], in the weights' floating-point type)."""
    return mean_pool_l2(hidden_states(w, n_layers, n_heads, ids, eps))


def encode_texts(w: Dict[str, np.ndarray], n_layers: int, n_heads: int,
                 tokens: np.ndarray, cu_seqlens: np.ndarray,
                 indices: Sequence[int], eps: float = 1e-12) -> np.ndarray:
    """Embeddings [len(indices), d] of the chosen texts, each encoded alone."""
    d = w["word_emb"].shape[1]
    out = np.empty((len(indices), d), dtype=w["word_emb"].dtype)
    for j, i in enumerate(indices):
        ids = tokens[int(cu_seqlens[i]):int(cu_seqlens[i + 1])]
        out[j] = encode_text(w, n_layers, n_heads, ids, eps)
    return out


def placement(part_offsets: np.ndarray, i: int):
    """(partition, row) of global text i: the unique p with
    part_offsets[p] <= i < part_offsets[p+1], and row i - part_offsets[p]."""
    offs = np.asarray(part_offsets)
    p = int(np.searchsorted(offs, i, side="right")) - 1
    return p, int(i - offs[p])


def encode_workload(w: Dict[str, np.ndarray], n_layers: int, n_heads: int,
                    tokens: np.ndarray, cu_seqlens: np.ndarray,
                    part_offsets: np.ndarray, eps: float = 1e-12) -> List[np.ndarray]:
    """Per-partition outputs: out[p][i - part_offsets[p]] = e_i for every text i."""
    d = w["word_emb"].shape[1]
    n_parts = len(part_offsets) - 1
    out = [np.empty((int(part_offsets[p + 1] - part_offsets[p]), d), dtype=w["word_emb"].dtype)
           for p in range(n_parts)]
    n = len(cu_seqlens) - 1
    for i in range(n):
        p, r = placement(part_offsets, i)
        ids = tokens[int(cu_seqlens[i]):int(cu_seqlens[i + 1])]
        out[p][r] = encode_text(w, n_layers, n_heads, ids, eps)
    return out

