"""Theorem 1 (IPC amortization) and the per-call cost tool, on the CPU.

The oracle's cost model is pinned to the paper's worked example (Sec. 4,
"Mixed regime": c_ipc = 0.087 s, c_enc = 0.149 ms, G = 4, P = 4,000,
N = 10^7, F = 100 gives alpha = 0.93 and a predicted speedup of 1.89) and to
the model's own definition summed call by call; the measurement tool's plans
and fit are checked against plain definitions.
"""
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import plan as OP
from paper_2605_01060_amd import callcost as CC
from paper_2605_01060_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "theorem1_example.json")


def test_theorem1_worked_example():
    g = json.load(open(GOLDEN))
    a = OP.ipc_alpha(g["P"], g["c_ipc_s"], g["N"], g["c_enc_s"], g["G"])
    assert a == pytest.approx(g["alpha"], abs=0.005)
    s = OP.ipc_speedup(a, g["F"], g["P"])
    assert s == pytest.approx(g["speedup_predicted"], abs=0.005)
    # the measured speedup the paper reports is within its stated 2 % error
    assert abs(s - g["speedup_measured"]) / g["speedup_measured"] < 0.02
    assert OP.ipc_threshold(0.087, 0.149e-3, 4) == pytest.approx(2336, rel=0.01)  # n* ~ 2,340


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(1, 5000), min_size=1, max_size=60), st.integers(1, 40),
       st.floats(1e-4, 1.0), st.floats(1e-7, 1e-3), st.integers(1, 8))
def test_theorem1_matches_call_by_call_sum(sizes, F, c_call, c_enc, G):
    """(1 + a)/(1 + a F/P) equals the ratio of the summed call times."""
    N, P = sum(sizes), len(sizes)
    t_pbp = OP.plan_time(sizes, c_call, c_enc, G)
    flush_sizes = [N // F + (1 if i < N % F else 0) for i in range(F)]
    t_surge = OP.plan_time(flush_sizes, c_call, c_enc, G)
    a = OP.ipc_alpha(P, c_call, N, c_enc, G)
    assert OP.ipc_speedup(a, F, P) == pytest.approx(t_pbp / t_surge, rel=1e-9)
    # the measurement tool's formula is the same function
    assert CC.ipc_speedup(a, F, P) == pytest.approx(OP.ipc_speedup(a, F, P), rel=1e-12)


def test_theorem1_limits():
    assert OP.ipc_speedup(0.0, 10, 1000) == 1.0
    assert OP.ipc_speedup(1e12, 10, 1000) == pytest.approx(100.0, rel=1e-6)  # -> P / F


def _covers_once(calls, part_offsets):
    n = int(part_offsets[-1])
    seen = np.zeros(n, np.int64)
    for t0, t1, segs in calls:
        assert sum(int(s["count"]) for s in segs) == t1 - t0
        for s in segs:
            p = int(s["partition"])
            g0 = t0 + int(s["first_text"])
            assert g0 == part_offsets[p] + int(s["row_offset"])
            assert g0 + int(s["count"]) <= part_offsets[p + 1]
            seen[g0:g0 + int(s["count"])] += 1
    assert np.all(seen == 1)


@pytest.mark.parametrize("chunk", [1, 7, 1000, 5000, 10 ** 6])
def test_fsb_plan(chunk):
    spec = W.WORKLOADS["minilm"]
    offs = W.make_workload(spec).part_offsets
    calls = CC.plan_fsb(offs, chunk)
    n = int(offs[-1])
    assert len(calls) == (n + chunk - 1) // chunk
    assert all(t1 - t0 == min(chunk, n - t0) for t0, t1, _ in calls)
    _covers_once(calls, offs)


def test_pbp_plan_one_call_per_partition():
    offs = np.array([0, 3, 3, 10, 11, 11, 40], np.int64)  # with empty partitions
    calls = CC.plan_pbp(offs)
    assert [(t0, t1) for t0, t1, _ in calls] == [(0, 3), (3, 10), (10, 11), (11, 40)]
    _covers_once(calls, offs)
    spec = W.WORKLOADS["bge"]
    offs = W.make_workload(spec).part_offsets
    calls = CC.plan_pbp(offs)
    assert len(calls) == int(np.count_nonzero(np.diff(offs)))
    _covers_once(calls, offs)


def test_surge_plan_matches_oracle():
    offs = W.make_workload(W.WORKLOADS["bge"]).part_offsets
    calls = CC.plan_surge(offs, 4096, 20000)
    ref = OP.plan(offs, 4096, 20000, OP.R2)
    assert [(t0, t1) for t0, t1, _ in calls] == [(s.text_begin, s.text_end) for s in ref]


def test_fit_call_cost_recovers_line():
    rng = np.random.default_rng(0)
    n = rng.integers(1, 20000, size=200)
    ms = 1.75 + n * 0.0123
    c0, c1 = CC.fit_call_cost(n, ms)
    assert c0 == pytest.approx(1.75, rel=1e-9) and c1 == pytest.approx(0.0123, rel=1e-9)
