"""Python binding of libsurge.so (ctypes), same names as the C-ABI.

Argument marshalling only: host arrays are passed as NumPy buffers, device
buffers as anything with ``data_ptr()`` (a torch tensor on the GPU) or a raw
integer address, streams as a ``torch.cuda.Stream`` / raw handle / None.
Every step of the encode path runs in the library's HIP kernels; if the
library is not built, loading it raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsurge.so")

SURGE_OK = 0
SURGE_ERR_INVALID_ARGUMENT = 1
SURGE_ERR_CAPACITY = 2
SURGE_ERR_OUT_OF_MEMORY = 3
SURGE_ERR_DEVICE = 4
SURGE_ERR_INTERNAL = 5

SURGE_POLICY_SPLIT = 0
SURGE_POLICY_LITERAL = 1

SURGE_WEIGHTS_F32 = 0
SURGE_WEIGHTS_BF16 = 1

KERNEL_NAMES = ["embed", "qkv", "attn", "oproj", "ln1", "ffn1", "ffn2", "ln2", "pool"]

SEGMENT_DTYPE = np.dtype([("first_text", "<i8"), ("count", "<i8"), ("row_offset", "<i8"),
                          ("partition", "<i4"), ("reserved", "<i4")])
SUPERBATCH_DTYPE = np.dtype([("text_begin", "<i8"), ("text_end", "<i8"),
                             ("seg_begin", "<i8"), ("seg_end", "<i8")])


class SurgeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"surge status {status}: {message}")
        self.status = status


class EncoderDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("vocab_size", ctypes.c_int32), ("max_positions", ctypes.c_int32),
                ("ln_eps", ctypes.c_float), ("weight_dtype", ctypes.c_int32)]


class StreamStats(ctypes.Structure):
    _fields_ = [("n_superbatches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("ttfo_ms", ctypes.c_double), ("enc_ms", ctypes.c_double),
                ("h2d_ms", ctypes.c_double), ("d2h_ms", ctypes.c_double),
                ("rho", ctypes.c_double), ("rho_measured", ctypes.c_double),
                ("staging_bytes", ctypes.c_int64), ("max_sb_texts", ctypes.c_int64),
                ("max_sb_tokens", ctypes.c_int64)]


class KernelStat(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


_lib = None

_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64

_SIGNATURES = {
    "surge_version": ([], ctypes.c_char_p),
    "surge_last_error": ([], ctypes.c_char_p),
    "surge_plan": ([_P, _I32, _I64, _I64, _I32, _P, _I64, _P, _P, _I64, _P], _I32),
    "surge_validate_superbatch": ([_P, _I64, _I64, _P, _P, _I64, _P, _P, _I32], _I32),
    "surge_validate_input": ([_P, _I64, _P, _P, _I32, _I64, _I64, _I32, _P, _P, _P, _P], _I32),
    "surge_encoder_create": ([_P, _P, _I32, _I64, _P], _I32),
    "surge_encoder_destroy": ([_P], None),
    "surge_encoder_info": ([_P, _P, _P, _P], _I32),
    "surge_encode_superbatch": ([_P, _I64, _I64, _P, _P, _P, _I64, _P, _P, _I32, _P], _I32),
    "surge_encode_all": ([_P, _I64, _P, _P, _P, _I32, _I64, _I64, _I32, _P, _I64, _P, _P], _I32),
    "surge_encode_all_streamed": ([_P, _I64, _P, _P, _P, _I32, _I64, _I64, _I32, _P, _I32, _P, _P,
                                   _P, _I64, _P], _I32),
    "surge_check": ([_P, _P], _I32),
    "surge_profile_enable": ([_P, _I32], _I32),
    "surge_profile_select": ([_P, ctypes.c_uint32], _I32),
    "surge_profile_read": ([_P, _P, _I32], _I32),
    "surge_op_embed_ln": ([_I64, _P, _P, _P, _I32, _P, _I32, _P, _P, ctypes.c_float, _I32, _P, _P], _I32),
    "surge_op_linear": ([_I64, _I32, _I32, _P, _P, _P, _P, _I32, _P, _P], _I32),
    "surge_op_linear_ln": ([_I64, _I32, _I32, _P, _P, _P, _P, _I32, _P, _I32, _P, _P, _P,
                            ctypes.c_float, _P, _P, _P], _I32),
    "surge_op_linear_ln_noalloc": ([_I64, _I32, _I32, _P, _P, _P, _P, _I32, _P, _I32, _P, _P,
                                    _P, ctypes.c_float, _P, _P, _P], _I32),
    "surge_op_linear_stats_width": ([_I64, _I32], _I32),
    "surge_op_attention": ([_I64, _P, _I32, _I32, _P, _P, _P], _I32),
    "surge_op_layernorm": ([_I64, _I32, _P, _P, _P, ctypes.c_float, _P, _P], _I32),
    "surge_op_pool_l2": ([_I64, _P, _I32, _P, _P, _P], _I32),
}


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2605_01060_amd.build`")
        l = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(l, name)
            fn.argtypes = args
            fn.restype = res
        _lib = l
    return _lib


def exported_symbols() -> List[str]:
    return list(_SIGNATURES)


def _check(status: int):
    if status != SURGE_OK:
        raise SurgeError(status, surge_last_error())


def _host(a: np.ndarray, dtype) -> Tuple[np.ndarray, int]:
    a = np.ascontiguousarray(a, dtype=dtype)
    return a, a.ctypes.data


def _dev(x) -> int:
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _hptr(x) -> int:
    """Address of a host buffer: a NumPy array or a CPU torch tensor."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        assert x.flags.c_contiguous
        return x.ctypes.data
    assert not x.is_cuda and x.is_contiguous()
    return int(x.data_ptr())


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def surge_version() -> str:
    return lib().surge_version().decode()


def surge_last_error() -> str:
    return lib().surge_last_error().decode()


def surge_plan(part_offsets, b_min: int, n_max: int = 0,
               policy: int = SURGE_POLICY_SPLIT) -> Tuple[np.ndarray, np.ndarray]:
    """SuperBatches and segments (structured arrays) of a CSR partition layout."""
    offs, p = _host(part_offsets, np.int64)
    n_parts = offs.shape[0] - 1
    ns, ng = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(lib().surge_plan(p, n_parts, b_min, n_max, policy, None, 0, ctypes.byref(ns),
                            None, 0, ctypes.byref(ng)))
    sbs = np.zeros(max(ns.value, 1), dtype=SUPERBATCH_DTYPE)
    segs = np.zeros(max(ng.value, 1), dtype=SEGMENT_DTYPE)
    _check(lib().surge_plan(p, n_parts, b_min, n_max, policy, sbs.ctypes.data, sbs.shape[0],
                            ctypes.byref(ns), segs.ctypes.data, segs.shape[0], ctypes.byref(ng)))
    return sbs[:ns.value], segs[:ng.value]


def make_desc(n_layers, d_model, n_heads, d_ff, vocab_size, max_positions,
              ln_eps=1e-12, weight_dtype=SURGE_WEIGHTS_F32) -> EncoderDesc:
    return EncoderDesc(n_layers, d_model, n_heads, d_ff, vocab_size, max_positions, ln_eps,
                       weight_dtype)


def segments_array(rows: Sequence[Tuple[int, int, int, int]]) -> np.ndarray:
    """Segment records from (first_text, count, partition, row_offset) tuples."""
    out = np.zeros(len(rows), dtype=SEGMENT_DTYPE)
    for i, (f, c, p, r) in enumerate(rows):
        out[i] = (f, c, r, p, 0)
    return out


def surge_validate_superbatch(desc: EncoderDesc, n_texts: int, n_tokens: int, cu_seqlens,
                              segments: np.ndarray, part_sizes, part_out_ptrs) -> int:
    """Status code of the host-side argument check (does not raise)."""
    cu, pcu = _host(cu_seqlens, np.int64)
    segs = np.ascontiguousarray(segments, dtype=SEGMENT_DTYPE)
    sizes, psz = _host(part_sizes, np.int64)
    outs, pout = _host(part_out_ptrs, np.uint64)
    return lib().surge_validate_superbatch(ctypes.byref(desc), n_texts, n_tokens, pcu,
                                           segs.ctypes.data if segs.size else None,
                                           segs.shape[0], psz, pout, sizes.shape[0])


def surge_validate_input(desc: EncoderDesc, n_texts: int, cu_seqlens, part_offsets, b_min: int,
                         n_max: int, policy: int, part_out_ptrs) -> Tuple[int, Dict[str, int]]:
    """Status code of the whole-input check (does not raise) and, on success,
    the plan's SuperBatch count and largest SuperBatch in texts and tokens."""
    cu, pcu = _host(cu_seqlens, np.int64)
    offs, poff = _host(part_offsets, np.int64)
    outs, pout = _host(part_out_ptrs, np.uint64)
    ns, mt, mk = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int64(0)
    st = lib().surge_validate_input(ctypes.byref(desc), n_texts, pcu, poff, offs.shape[0] - 1,
                                    b_min, n_max, policy, pout, ctypes.byref(ns),
                                    ctypes.byref(mt), ctypes.byref(mk))
    return st, {"n_superbatches": ns.value, "max_sb_texts": mt.value, "max_sb_tokens": mk.value}


def surge_encoder_create(desc: EncoderDesc, weights: Sequence[np.ndarray],
                         max_tokens_per_chunk: int) -> int:
    """weights: float32 arrays (desc.weight_dtype = F32) or uint16 arrays of
    bf16 bit patterns (BF16), in the fixed order."""
    dt = np.float32 if desc.weight_dtype == SURGE_WEIGHTS_F32 else np.uint16
    arrs = [np.ascontiguousarray(w, dtype=dt) for w in weights]
    ptrs = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    h = ctypes.c_void_p(0)
    _check(lib().surge_encoder_create(ctypes.byref(desc), ptrs, len(arrs), max_tokens_per_chunk,
                                      ctypes.byref(h)))
    return h.value


def surge_encoder_destroy(handle: int):
    lib().surge_encoder_destroy(handle)


def surge_encoder_info(handle: int) -> Tuple[EncoderDesc, int, int]:
    d = EncoderDesc()
    mt, wb = ctypes.c_int64(0), ctypes.c_int64(0)
    _check(lib().surge_encoder_info(handle, ctypes.byref(d), ctypes.byref(mt), ctypes.byref(wb)))
    return d, mt.value, wb.value


def surge_encode_superbatch(handle: int, n_texts: int, n_tokens: int, d_token_ids, cu_seqlens,
                            segments: np.ndarray, part_out_ptrs, part_sizes, stream=None):
    cu, pcu = _host(cu_seqlens, np.int64)
    segs = np.ascontiguousarray(segments, dtype=SEGMENT_DTYPE)
    outs, pout = _host(part_out_ptrs, np.uint64)
    sizes, psz = _host(part_sizes, np.int64)
    _check(lib().surge_encode_superbatch(handle, n_texts, n_tokens, _dev(d_token_ids), pcu,
                                         segs.ctypes.data if segs.size else None, segs.shape[0],
                                         pout, psz, outs.shape[0], _stream(stream)))


def surge_encode_all(handle: int, n_texts: int, d_token_ids, cu_seqlens, part_offsets,
                     b_min: int, n_max: int, policy: int, part_out_ptrs, first_sb: int = 0,
                     stream=None) -> int:
    cu, pcu = _host(cu_seqlens, np.int64)
    offs, poff = _host(part_offsets, np.int64)
    outs, pout = _host(part_out_ptrs, np.uint64)
    nsb = ctypes.c_int64(0)
    _check(lib().surge_encode_all(handle, n_texts, _dev(d_token_ids), pcu, poff, offs.shape[0] - 1,
                                  b_min, n_max, policy, pout, first_sb, ctypes.byref(nsb),
                                  _stream(stream)))
    return nsb.value



def surge_encode_all_streamed(handle: int, n_texts: int, h_token_ids, cu_seqlens, part_offsets,
                              b_min: int, n_max: int, policy: int, h_out, overlap: int,
                              compute_stream=None, copy_stream=None,
                              sb_times: Optional[np.ndarray] = None) -> Dict[str, float]:
    """h_token_ids / h_out: host buffers (pinned torch CPU tensors or NumPy
    arrays; pass pinned memory for overlapping copies).  overlap: 0 in order
    on compute_stream, 1 copies on copy_stream, 2 zero copy (h_out must be
    pinned).  Returns the timing summary; per-SuperBatch (upload, encode,
    download) ms go to sb_times [cap, 3] float64 if given."""
    cu, pcu = _host(cu_seqlens, np.int64)
    offs, poff = _host(part_offsets, np.int64)
    st = StreamStats()
    cap = 0 if sb_times is None else int(sb_times.shape[0])
    pt = 0 if sb_times is None else sb_times.ctypes.data
    if sb_times is not None:
        assert sb_times.dtype == np.float64 and sb_times.flags.c_contiguous and sb_times.shape[1:] == (3,)
    _check(lib().surge_encode_all_streamed(handle, n_texts, _hptr(h_token_ids), pcu, poff,
                                           offs.shape[0] - 1, b_min, n_max, policy, _hptr(h_out),
                                           overlap, _stream(compute_stream), _stream(copy_stream),
                                           pt, cap, ctypes.byref(st)))
    return {k: getattr(st, k) for k, _ in StreamStats._fields_}

def surge_check(handle: int, stream=None):
    _check(lib().surge_check(handle, _stream(stream)))


def surge_profile_enable(handle: int, on: bool):
    _check(lib().surge_profile_enable(handle, 1 if on else 0))


def surge_profile_select(handle: int, kinds: Sequence[str]):
    """Time only the launches of the named kernel classes (empty: none)."""
    mask = 0
    for k in kinds:
        mask |= 1 << KERNEL_NAMES.index(k)
    _check(lib().surge_profile_select(handle, mask))


def surge_profile_read(handle: int) -> Dict[str, Dict[str, float]]:
    stats = (KernelStat * len(KERNEL_NAMES))()
    _check(lib().surge_profile_read(handle, stats, len(KERNEL_NAMES)))
    return {n: {"launches": s.launches, "total_ms": s.total_ms, "flops": s.flops,
                "bytes": s.bytes} for n, s in zip(KERNEL_NAMES, stats)}


# Stage-level entry points --------------------------------------------------

def surge_op_embed_ln(cu_seqlens, d_tokens, d_word, vocab, d_pos, max_pos, d_gamma, d_beta,
                      eps, d, d_out, stream=None):
    cu, pcu = _host(cu_seqlens, np.int64)
    _check(lib().surge_op_embed_ln(cu.shape[0] - 1, pcu, _dev(d_tokens), _dev(d_word), vocab,
                                   _dev(d_pos), max_pos, _dev(d_gamma), _dev(d_beta), eps, d,
                                   _dev(d_out), _stream(stream)))


def surge_op_linear(M, N, K, d_x, d_w, d_bias, d_res, epilogue, d_y, stream=None):
    _check(lib().surge_op_linear(M, N, K, _dev(d_x), _dev(d_w), _dev(d_bias), _dev(d_res),
                                 epilogue, _dev(d_y), _stream(stream)))


def surge_op_linear_ln(M, N, K, x, w, bias, res, epilogue, stats_in, parts_in, col_s, gamma,
                       beta, eps, stats_out, y, stream=None):
    _check(lib().surge_op_linear_ln(M, N, K, _dev(x), _dev(w), _dev(bias), _dev(res), epilogue,
                                    _dev(stats_in), parts_in, _dev(col_s), _dev(gamma),
                                    _dev(beta), eps, _dev(stats_out), _dev(y), _stream(stream)))


def surge_op_linear_ln_noalloc(M, N, K, x, w, bias, res, epilogue, stats_in, parts_in, col_s,
                               gamma, beta, eps, stats_out, y, stream=None):
    """As surge_op_linear_ln, with the row factors in the library's static
    scratch; only enqueues on `stream`."""
    _check(lib().surge_op_linear_ln_noalloc(M, N, K, _dev(x), _dev(w), _dev(bias), _dev(res),
                                            epilogue, _dev(stats_in), parts_in, _dev(col_s),
                                            _dev(gamma), _dev(beta), eps, _dev(stats_out), _dev(y),
                                            _stream(stream)))


def surge_op_linear_stats_width(M: int, N: int) -> int:
    return int(lib().surge_op_linear_stats_width(M, N))


def surge_op_attention(cu_seqlens, n_heads, d_head, d_qkv, d_out, stream=None):
    cu, pcu = _host(cu_seqlens, np.int64)
    _check(lib().surge_op_attention(cu.shape[0] - 1, pcu, n_heads, d_head, _dev(d_qkv),
                                    _dev(d_out), _stream(stream)))


def surge_op_layernorm(M, d, d_x, d_gamma, d_beta, eps, d_y, stream=None):
    _check(lib().surge_op_layernorm(M, d, _dev(d_x), _dev(d_gamma), _dev(d_beta), eps, _dev(d_y),
                                    _stream(stream)))


def surge_op_pool_l2(cu_seqlens, d, d_x, d_out, stream=None):
    cu, pcu = _host(cu_seqlens, np.int64)
    _check(lib().surge_op_pool_l2(cu.shape[0] - 1, pcu, d, _dev(d_x), _dev(d_out),
                                  _stream(stream)))


# Convenience: an encoder object over device-resident inputs ----------------

class Encoder:
    """Owns a surge_encoder; weights are the fp32 arrays of the fixed order."""

    def __init__(self, desc: EncoderDesc, weights: Sequence[np.ndarray],
                 max_tokens_per_chunk: int = 1 << 20):
        self.desc = desc
        self.handle = surge_encoder_create(desc, weights, max_tokens_per_chunk)

    def close(self):
        if self.handle:
            surge_encoder_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def encode_all(self, n_texts, d_tokens, cu_seqlens, part_offsets, b_min, n_max,
                   part_out_ptrs, policy=SURGE_POLICY_SPLIT, first_sb=0, stream=None) -> int:
        return surge_encode_all(self.handle, n_texts, d_tokens, cu_seqlens, part_offsets, b_min,
                                n_max, policy, part_out_ptrs, first_sb, stream)

    def encode_all_streamed(self, n_texts, h_tokens, cu_seqlens, part_offsets, b_min, n_max,
                            h_out, overlap=2, compute_stream=None, copy_stream=None,
                            policy=SURGE_POLICY_SPLIT, sb_times=None) -> Dict[str, float]:
        return surge_encode_all_streamed(self.handle, n_texts, h_tokens, cu_seqlens, part_offsets,
                                         b_min, n_max, policy, h_out, overlap, compute_stream,
                                         copy_stream, sb_times)

    def encode_superbatch(self, n_texts, n_tokens, d_tokens, cu_seqlens, segments,
                          part_out_ptrs, part_sizes, stream=None):
        surge_encode_superbatch(self.handle, n_texts, n_tokens, d_tokens, cu_seqlens, segments,
                                part_out_ptrs, part_sizes, stream)

    def check(self, stream=None):
        surge_check(self.handle, stream)

    def profile(self, on: bool, kinds: Optional[Sequence[str]] = None):
        if on and kinds is not None:
            surge_profile_select(self.handle, kinds)
        else:
            surge_profile_enable(self.handle, on)

    def profile_read(self):
        return surge_profile_read(self.handle)
