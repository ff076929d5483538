"""Helpers shared by the GPU parity tests (not a test module)."""
from __future__ import annotations

import json
import os

import numpy as np

from paper_2605_01060_amd import surge as S
from paper_2605_01060_amd import workload as W

# Acceptance bar for end-to-end embeddings (bf16 compute vs the fp32 oracle):
# per-text cosine >= 0.9995 and max-abs <= 2e-2 per component, exact placement.
COS_MIN = 0.9995
MAXABS = 2e-2
# Supplementary: cosine after removing the oracle's mean embedding over the
# compared texts (bf16 noise is amplified by how alike random-init
# embeddings are, so the bound depends on depth and width).  The bounds come
# from a bf16 simulation of the oracle over 120 texts per encoder shape,
# written by tests/golden/derive_centred_bounds.py.
with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                       "centred_bounds.json")) as _f:
    CENTRED_MIN = json.load(_f)["configs"]


def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    return torch


def desc_of(shape: W.EncoderShape) -> S.EncoderDesc:
    return S.make_desc(shape.n_layers, shape.d_model, shape.n_heads, shape.d_ff,
                       shape.vocab_size, shape.max_positions, shape.ln_eps)


def weight_list(shape: W.EncoderShape, weights):
    return [weights[n] for n in W.weight_names(shape.n_layers)]


def cosine_rows(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return (a * b).sum(1) / (np.linalg.norm(a, axis=1) * np.linalg.norm(b, axis=1))


def compare_embeddings(got: np.ndarray, ref: np.ndarray, config: str):
    cos = cosine_rows(got, ref)
    maxabs = float(np.max(np.abs(got.astype(np.float64) - ref)))
    mu = ref.mean(axis=0, keepdims=True)
    ccos = cosine_rows(got - mu, ref - mu) if ref.shape[0] > 1 else cos
    return {"cos_min": float(cos.min()), "maxabs": maxabs, "centred_min": float(ccos.min()),
            "n": int(ref.shape[0])}


def assert_parity(got: np.ndarray, ref: np.ndarray, config: str):
    st = compare_embeddings(got, ref, config)
    print(f"[parity {config}] {st}", flush=True)
    assert st["cos_min"] >= COS_MIN, st
    assert st["maxabs"] <= MAXABS, st
    if st["n"] > 1:
        assert st["centred_min"] >= CENTRED_MIN[config], st
    return st
