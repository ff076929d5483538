"""Derive the supplementary centred-cosine bounds of the GPU parity tests.

    python tests/golden/derive_centred_bounds.py   # writes centred_bounds.json

The GPU path computes in bf16 with fp32 accumulation; the parity tests hold
it to the float32 oracle with per-text cosine >= 0.9995 and max-abs <= 2e-2,
and additionally compare *centred* embeddings (the oracle's mean over the
compared texts removed), which removes the component that random-init
embeddings share and so amplifies bf16 noise by how alike the texts are.  A
single bound does not fit every encoder depth and width, so each one is
derived here from a bf16 simulation of the oracle:

* weights rounded to bf16 (nearest, ties to even);
* the activations rounded to bf16 at every point where the GPU path stores
  them between kernels: the embedding LayerNorm output, Q|K|V, the softmax
  probabilities before the P V product, the attention output, each residual
  sum and LayerNorm output, the GELU output; fp32 everywhere else;
* every computation step is the oracle's own (``oracle.encoder``).

For each encoder shape, 120 texts (the first texts of the configuration's
workload) are simulated and compared with the float32 oracle; the centred
cosine is taken over the whole set and over every run of 8 consecutive texts
(the smallest sets the GPU tests compare).  The bound is
1 - 4 (1 - worst simulated centred cosine): a margin of 4x for the GPU's own
rounding points, which differ in detail (LayerNorms folded into the GEMMs).

To show the bound still has teeth, the same comparison is made for a copy of
the oracle with a planted mistake (attention across the boundary between two
consecutive texts, i.e. a missing block-diagonal mask), which a correct bound
must reject.
"""
from __future__ import annotations

import json
import math
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import encoder as E  # noqa: E402
from paper_2605_01060_amd import workload as W  # noqa: E402

N_TEXTS = 120
RUN = 8
MARGIN = 4.0
SHAPES = {"tiny": ["tiny"], "minilm": ["minilm", "minilm_heavy"], "bge": ["bge", "bge_s1"],
          "large": ["large"]}


def bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value of each float32 (ties to even), as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def attention_bf16(qkv: np.ndarray, n_heads: int) -> np.ndarray:
    """The oracle's per-head attention with P rounded to bf16 before P V."""
    L, three_d = qkv.shape
    d = three_d // 3
    dh = d // n_heads
    out = np.empty((L, d), dtype=np.float32)
    for h in range(n_heads):
        c = slice(h * dh, (h + 1) * dh)
        p = E.softmax_rows(qkv[:, c] @ qkv[:, d:2 * d][:, c].T / math.sqrt(dh))
        out[:, c] = bf16(p) @ qkv[:, 2 * d:][:, c]
    return out


def hidden_bf16(w, n_layers: int, n_heads: int, ids: np.ndarray, eps: float) -> np.ndarray:
    x = bf16(E.embed(w, ids, eps))
    for l in range(n_layers):
        p = f"layer{l}."
        qkv = bf16(E.linear(x, w[p + "w_qkv"], w[p + "b_qkv"]))
        a = bf16(attention_bf16(qkv, n_heads))
        r = bf16(x + E.linear(a, w[p + "w_o"], w[p + "b_o"]))
        x = bf16(E.layer_norm(r, w[p + "ln1_g"], w[p + "ln1_b"], eps))
        hdn = bf16(E.gelu(E.linear(x, w[p + "w_1"], w[p + "b_1"])))
        r = bf16(x + E.linear(hdn, w[p + "w_2"], w[p + "b_2"]))
        x = bf16(E.layer_norm(r, w[p + "ln2_g"], w[p + "ln2_b"], eps))
    return x


def leaky_pair(w, n_layers: int, n_heads: int, ids_a, ids_b, eps: float) -> np.ndarray:
    """Planted mistake: text a encoded with text b's tokens visible to its
    attention (one packed sequence, positions restarting per text, no mask);
    returns text a's embedding."""
    La = len(ids_a)
    x = np.concatenate([E.embed(w, ids_a, eps), E.embed(w, ids_b, eps)])
    for l in range(n_layers):
        x = E.encoder_layer(w, l, x, n_heads, eps)
    return E.mean_pool_l2(x[:La])


def centred_min(got: np.ndarray, ref: np.ndarray) -> float:
    """Worst per-text cosine after removing the reference mean, over the whole
    set and over every run of RUN consecutive texts."""
    got = got.astype(np.float64)
    ref = ref.astype(np.float64)

    def one(g, r):
        mu = r.mean(axis=0, keepdims=True)
        a, b = g - mu, r - mu
        return float(((a * b).sum(1) / (np.linalg.norm(a, axis=1) *
                                        np.linalg.norm(b, axis=1))).min())

    vals = [one(got, ref)]
    for s in range(0, got.shape[0] - RUN + 1, RUN):
        vals.append(one(got[s:s + RUN], ref[s:s + RUN]))
    return min(vals)


def derive(shape_name: str) -> dict:
    spec = W.WORKLOADS[shape_name]
    sh = spec.encoder
    wl = W.make_workload(spec)
    w32 = E.as_f32(W.make_weights(sh, seed=spec.seed))
    wb = {k: bf16(v) for k, v in w32.items()}
    idx = list(range(N_TEXTS))
    ref = E.encode_texts(w32, sh.n_layers, sh.n_heads, wl.tokens, wl.cu_seqlens, idx, sh.ln_eps)
    sim = np.stack([E.mean_pool_l2(hidden_bf16(wb, sh.n_layers, sh.n_heads,
                                               wl.tokens[wl.cu_seqlens[i]:wl.cu_seqlens[i + 1]],
                                               sh.ln_eps)) for i in idx])
    cos = ((sim.astype(np.float64) * ref).sum(1) /
           (np.linalg.norm(sim.astype(np.float64), axis=1) * np.linalg.norm(ref, axis=1)))
    cmin = centred_min(sim, ref)
    bound = 1.0 - MARGIN * (1.0 - cmin)
    out = {"n_texts": N_TEXTS, "sim_cos_min": float(cos.min()),
           "sim_maxabs": float(np.abs(sim.astype(np.float64) - ref).max()),
           "sim_centred_min": cmin, "bound": bound}
    if shape_name in ("tiny", "bge"):
        n_leak = 24
        toks = [wl.tokens[wl.cu_seqlens[i]:wl.cu_seqlens[i + 1]] for i in range(n_leak + 1)]
        leak = np.stack([leaky_pair(w32, sh.n_layers, sh.n_heads, toks[i], toks[i + 1], sh.ln_eps)
                         for i in range(n_leak)])
        out["leak_centred_min"] = centred_min(leak, ref[:n_leak])
        out["leak_rejected"] = out["leak_centred_min"] < bound
    print(shape_name, out, flush=True)
    return out


def main() -> int:
    res = {"script": "tests/golden/derive_centred_bounds.py", "margin": MARGIN, "run": RUN,
           "shapes": {}, "configs": {}}
    for shape_name, configs in SHAPES.items():
        r = derive(shape_name)
        res["shapes"][shape_name] = r
        for c in configs:
            res["configs"][c] = r["bound"]
    with open(os.path.join(HERE, "centred_bounds.json"), "w") as f:
        json.dump(res, f, indent=1)
        f.write("\n")
    return 0


if __name__ == "__main__":
    sys.exit(main())
