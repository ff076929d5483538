"""The C-ABI on the CPU: the library loads, exports every declared symbol,
its planner matches the planner oracle, and host validation rejects each
malformed input with the documented status."""
import ctypes
import glob
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import plan as OP
from paper_2605_01060_amd import surge as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for h in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))):
        text = open(h).read()
        names += re.findall(r"^\s*(?:surge_status|void|int32_t|const char\*)\s+(surge_\w+)\s*\(", text,
                            re.M)
    return names


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 17
    lib = S.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(S.exported_symbols())


def test_version():
    assert re.match(r"^\d+\.\d+\.\d+$", S.surge_version())


def _oracle_flat(offsets, b_min, cap, policy):
    sbs = OP.plan(offsets, b_min, cap, OP.R1 if policy == S.SURGE_POLICY_LITERAL else OP.R2)
    return OP.flatten(sbs)


@settings(max_examples=300, deadline=None)
@given(sizes=st.lists(st.integers(0, 60), min_size=0, max_size=60),
       b_min=st.integers(1, 100), cap=st.integers(-1, 120),
       policy=st.sampled_from([S.SURGE_POLICY_SPLIT, S.SURGE_POLICY_LITERAL]))
def test_plan_matches_oracle(sizes, b_min, cap, policy):
    offs = np.concatenate([[0], np.cumsum(np.asarray(sizes, np.int64))]).astype(np.int64)
    sbs, segs = S.surge_plan(offs, b_min, cap, policy)
    ref_sb, ref_seg = _oracle_flat(offs, b_min, cap, policy)
    assert [tuple(int(v) for v in r) for r in sbs] == ref_sb
    assert [(int(r["first_text"]), int(r["count"]), int(r["partition"]), int(r["row_offset"]))
            for r in segs] == ref_seg


@pytest.mark.parametrize("name", ["bge", "minilm_heavy", "large"])
def test_plan_matches_oracle_on_workloads(name):
    from paper_2605_01060_amd import workload as W
    spec = W.WORKLOADS[name]
    rng = W._streams(spec.seed)[0]
    sizes = W.partition_sizes(rng, spec.n_texts, spec.n_parts, spec.part_sigma)
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    for policy in (S.SURGE_POLICY_SPLIT, S.SURGE_POLICY_LITERAL):
        sbs, segs = S.surge_plan(offs, spec.b_min, spec.n_max, policy)
        ref_sb, ref_seg = _oracle_flat(offs, spec.b_min, spec.n_max, policy)
        assert [tuple(int(v) for v in r) for r in sbs] == ref_sb
        assert len(segs) == len(ref_seg)


def test_plan_capacity_and_query():
    lib = S.lib()
    offs = np.array([0, 3, 7, 9], np.int64)
    ns, ng = ctypes.c_int64(0), ctypes.c_int64(0)
    assert lib.surge_plan(offs.ctypes.data, 3, 4, 0, 0, None, 0, ctypes.byref(ns), None, 0,
                          ctypes.byref(ng)) == S.SURGE_OK
    assert (ns.value, ng.value) == (2, 3)
    sbs = np.zeros(1, dtype=S.SUPERBATCH_DTYPE)
    segs = np.zeros(3, dtype=S.SEGMENT_DTYPE)
    st_ = lib.surge_plan(offs.ctypes.data, 3, 4, 0, 0, sbs.ctypes.data, 1, ctypes.byref(ns),
                         segs.ctypes.data, 3, ctypes.byref(ng))
    assert st_ == S.SURGE_ERR_CAPACITY
    assert np.all(sbs["text_end"] == 0)  # nothing written


@pytest.mark.parametrize("offs,b_min,policy", [
    ([1, 3], 1, 0),        # part_offsets[0] != 0
    ([0, 3, 2], 1, 0),     # decreasing
    ([0, 3], 0, 0),        # b_min < 1
    ([0, 3], 1, 7),        # unknown policy
])
def test_plan_rejects(offs, b_min, policy):
    with pytest.raises(S.SurgeError) as ei:
        S.surge_plan(np.array(offs, np.int64), b_min, 0, policy)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT


DESC = S.make_desc(2, 128, 2, 512, 30522, 64)


def _valid():
    cu = np.array([0, 3, 10, 12], np.int64)
    segs = S.segments_array([(0, 2, 0, 1), (2, 1, 1, 0)])
    sizes = np.array([3, 1], np.int64)
    outs = np.array([4096, 8192], np.uint64)
    return cu, segs, sizes, outs


def test_validate_accepts_valid_superbatch():
    cu, segs, sizes, outs = _valid()
    assert S.surge_validate_superbatch(DESC, 3, 12, cu, segs, sizes, outs) == S.SURGE_OK
    assert S.surge_validate_superbatch(DESC, 0, 0, np.zeros(1, np.int64),
                                       np.zeros(0, S.SEGMENT_DTYPE), sizes, outs) == S.SURGE_OK


def _mutations():
    out = []
    cu, segs, sizes, outs = _valid()
    c = cu.copy(); c[1] = 0; out.append(("zero-length text", c, segs, sizes, outs, 3, 12))
    c = cu.copy(); c[2] = c[1] + 65; c[3] = c[2] + 2
    out.append(("text longer than max_positions", c, segs, sizes, outs, 3, int(c[3])))
    c = cu.copy(); c[0] = 1; out.append(("cu[0] != 0", c, segs, sizes, outs, 3, 12))
    c = cu.copy(); c[2] = 2; out.append(("non-monotone cu", c, segs, sizes, outs, 3, 12))
    out.append(("n_tokens mismatch", cu, segs, sizes, outs, 3, 13))
    s = segs.copy(); s[1]["first_text"] = 1; out.append(("gap/overlap", cu, s, sizes, outs, 3, 12))
    s = segs.copy(); s[1]["count"] = 0; out.append(("empty segment", cu, s, sizes, outs, 3, 12))
    s = segs.copy(); s[1]["partition"] = 2; out.append(("partition out of range", cu, s, sizes, outs, 3, 12))
    s = segs.copy(); s[0]["row_offset"] = 2; out.append(("segment overflows partition", cu, s, sizes, outs, 3, 12))
    s = segs.copy(); s[0]["row_offset"] = -1; out.append(("negative row offset", cu, s, sizes, outs, 3, 12))
    o = outs.copy(); o[1] = 0; out.append(("NULL output", cu, segs, sizes, o, 3, 12))
    s = segs[:1].copy(); out.append(("segments do not cover texts", cu, s, sizes, outs, 3, 12))
    out.append(("negative n_texts", cu, segs, sizes, outs, -1, 12))
    return out


@pytest.mark.parametrize("case", _mutations(), ids=lambda c: c[0])
def test_validate_rejects(case):
    _, cu, segs, sizes, outs, n, T = case
    assert S.surge_validate_superbatch(DESC, n, T, cu, segs, sizes, outs) == \
        S.SURGE_ERR_INVALID_ARGUMENT
    assert S.surge_last_error()


@pytest.mark.parametrize("field,value", [("d_model", 96), ("n_heads", 5), ("d_ff", 100),
                                         ("n_layers", 0), ("max_positions", 0),
                                         ("weight_dtype", 2), ("d_model", 2048)])
def test_validate_rejects_bad_desc(field, value):
    d = S.make_desc(2, 128, 2, 512, 30522, 64)
    setattr(d, field, value)
    cu, segs, sizes, outs = _valid()
    assert S.surge_validate_superbatch(d, 3, 12, cu, segs, sizes, outs) == \
        S.SURGE_ERR_INVALID_ARGUMENT


def test_encoder_create_rejects_bad_arguments_without_touching_the_device():
    d = S.make_desc(2, 128, 2, 512, 30522, 64)
    with pytest.raises(S.SurgeError) as ei:
        S.surge_encoder_create(d, [np.zeros(1, np.float32)] * 3, 1024)
    assert ei.value.status == S.SURGE_ERR_INVALID_ARGUMENT


def test_validate_input_beyond_2_31_tokens():
    """The whole-input check keeps offsets in int64 and caps only each
    SuperBatch: 2^23 texts of 512 tokens (2^32 tokens in all) in 1,024
    partitions pass; a plan whose single SuperBatch reaches 2^31 tokens does
    not.  Only cu_seqlens and part_offsets exist; no token is allocated."""
    desc = S.make_desc(12, 768, 12, 3072, 30522, 512)
    n = 1 << 23
    cu = np.arange(n + 1, dtype=np.int64) * 512
    assert cu[-1] == 1 << 32
    offs = np.arange(1025, dtype=np.int64) * (n // 1024)
    outs = np.full(1024, 4096, dtype=np.uint64)  # never dereferenced
    st, info = S.surge_validate_input(desc, n, cu, offs, 4096, 20000, S.SURGE_POLICY_SPLIT, outs)
    assert st == S.SURGE_OK, S.surge_last_error()
    assert info == {"n_superbatches": 1024, "max_sb_texts": 8192, "max_sb_tokens": 8192 * 512}
    # one SuperBatch of 2^22 + 1 texts of 512 tokens: 2^31 + 512 tokens
    m = (1 << 22) + 1
    st, _ = S.surge_validate_input(desc, m, cu[:m + 1], np.array([0, m], np.int64), 1 << 30, 0,
                                   S.SURGE_POLICY_SPLIT, outs[:1])
    assert st == S.SURGE_ERR_INVALID_ARGUMENT
    assert "2^31" in S.surge_last_error()


def test_validate_input_rejects_and_accepts():
    desc = S.make_desc(2, 128, 2, 512, 30522, 64)
    cu = np.array([0, 3, 5, 9, 10], np.int64)
    offs = np.array([0, 2, 2, 4], np.int64)  # partition 1 is empty
    outs = np.array([4096, 0, 8192], np.uint64)  # an empty partition may have no output
    ok, info = S.surge_validate_input(desc, 4, cu, offs, 2, 0, S.SURGE_POLICY_SPLIT, outs)
    assert ok == S.SURGE_OK and info["n_superbatches"] == 2 and info["max_sb_tokens"] == 5
    bad = [
        (desc, 4, cu, offs, 2, 0, S.SURGE_POLICY_SPLIT, np.array([4096, 0, 0], np.uint64)),
        (desc, 4, np.array([0, 3, 3, 9, 10], np.int64), offs, 2, 0, 0, outs),  # empty text
        (desc, 4, np.array([0, 3, 5, 70, 71], np.int64), offs, 2, 0, 0, outs),  # > max_positions
        (desc, 4, np.array([1, 3, 5, 9, 10], np.int64), offs, 2, 0, 0, outs),  # cu[0] != 0
        (desc, 5, np.array([0, 3, 5, 9, 10, 11], np.int64), offs, 2, 0, 0, outs),  # offs end
        (desc, 4, cu, np.array([0, 3, 2, 4], np.int64), 2, 0, 0, outs),  # decreasing
        (desc, 4, cu, offs, 0, 0, 0, outs),  # b_min < 1
        (desc, 4, cu, offs, 2, 0, 7, outs),  # policy
    ]
    for args in bad:
        st, _ = S.surge_validate_input(*args)
        assert st == S.SURGE_ERR_INVALID_ARGUMENT, args
        assert S.surge_last_error()
