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


# --- PB-PBP-LB (FFD) and Lemma 1 -------------------------------------------

FFD_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "ffd_cases.json")


def test_ffd_golden():
    for c in json.load(open(FFD_GOLDEN))["cases"]:
        assert OP.ffd_pack(c["sizes"], c["capacity"]) == c["batches"]
        assert CC.ffd_batches(c["sizes"], c["capacity"]) == c["batches"]


def _opt_bins(sizes, cap):
    """Fewest bins by exhaustive search (tiny inputs)."""
    items = sorted([s for s in sizes if s > 0], reverse=True)
    best = [len(items)]

    def rec(i, loads):
        if len(loads) >= best[0]:
            return
        if i == len(items):
            best[0] = len(loads)
            return
        seen = set()
        for b in range(len(loads)):
            if loads[b] + items[i] <= cap and loads[b] not in seen:
                seen.add(loads[b])
                loads[b] += items[i]
                rec(i + 1, loads)
                loads[b] -= items[i]
        loads.append(items[i])
        rec(i + 1, loads)
        loads.pop()

    rec(0, [])
    return best[0]


@settings(max_examples=150, deadline=None)
@given(st.lists(st.integers(0, 10), min_size=1, max_size=9), st.integers(10, 14))
def test_ffd_invariants_and_bound(sizes, cap):
    bins = OP.ffd_pack(sizes, cap)
    flat = sorted(p for b in bins for p in b)
    assert flat == [p for p, n in enumerate(sizes) if n > 0]  # every partition once, whole
    assert all(sum(sizes[p] for p in b) <= cap for b in bins)
    # the FFD guarantee (Dósa 2007): FFD <= 11/9 OPT + 6/9
    opt = _opt_bins(sizes, cap)
    assert len(bins) <= 11 / 9 * opt + 6 / 9 + 1e-9
    assert CC.ffd_batches(sizes, cap) == bins


def test_ffd_oversized_partition_alone():
    bins = OP.ffd_pack([3, 25, 4, 30], 10)
    assert bins[0] == [3] and bins[1] == [1]  # never split, one batch each
    assert CC.ffd_batches([3, 25, 4, 30], 10) == bins


def test_plan_ffd_layout():
    wl = W.make_workload(W.WORKLOADS["minilm"])
    calls, perm, cu = CC.plan_ffd(wl.part_offsets, wl.cu_seqlens, 3000)
    assert sorted(perm.tolist()) == list(range(wl.n_texts))
    assert cu[-1] == wl.n_tokens
    lens = np.diff(wl.cu_seqlens)
    assert np.array_equal(np.diff(cu), lens[perm])
    for t0, t1, segs in calls:
        for s in segs:
            p = int(s["partition"])
            assert s["row_offset"] == 0 and s["count"] == wl.part_offsets[p + 1] - wl.part_offsets[p]
            a = t0 + int(s["first_text"])
            assert np.array_equal(perm[a:a + int(s["count"])],
                                  np.arange(wl.part_offsets[p], wl.part_offsets[p + 1]))
    tp = CC.permuted_tokens(wl.tokens, wl.cu_seqlens, perm)
    for k in (0, 17, wl.n_texts - 1):
        t = perm[k]
        assert np.array_equal(tp[cu[k]:cu[k + 1]], wl.tokens[wl.cu_seqlens[t]:wl.cu_seqlens[t + 1]])


def test_adversarial_order():
    sizes = np.array([50, 3, 900, 7, 2, 40, 5])
    order = CC.adversarial_order(sizes, 20)
    assert sorted(order.tolist()) == list(range(sizes.size))
    k = order.tolist().index(2)
    assert sizes[order[:k]].sum() < 20 and k > 0  # a buffer just short of B_min, then the largest
    assert OP.plan([0] + np.cumsum(sizes[order]).tolist(), 20, 0, OP.R1)[0].n_texts == \
        sizes[order[:k + 1]].sum()


@settings(max_examples=100, deadline=None)
@given(st.lists(st.integers(0, 400), min_size=1, max_size=40), st.integers(1, 300),
       st.integers(1, 600))
def test_lemma1_bound(sizes, b_min, cap):
    """Largest SuperBatch: R1 <= (B_min - 1) + n_max, R2 <= cap; both in
    every arrival order, including the adversarial one."""
    sizes = np.array(sizes)
    n_big = int(sizes.max())
    for order in (np.arange(sizes.size), CC.adversarial_order(sizes, b_min)):
        offs = [0] + np.cumsum(sizes[order]).tolist()
        r1 = max([sb.n_texts for sb in OP.plan(offs, b_min, 0, OP.R1)] + [0])
        r2 = max([sb.n_texts for sb in OP.plan(offs, b_min, cap, OP.R2)] + [0])
        assert r1 <= b_min - 1 + n_big
        assert r2 <= cap
        assert r1 <= OP.largest_superbatch_bound(b_min, n_big, 0, OP.R1)
        assert r2 <= OP.largest_superbatch_bound(b_min, n_big, cap, OP.R2)
        # M(S) grows with S, so the bound on S bounds the memory too (Lemma 1)
        assert OP.superbatch_memory(r2, 47, 384) <= OP.superbatch_memory(
            OP.largest_superbatch_bound(b_min, n_big, cap, OP.R2), 47, 384)


def test_lemma1_table_heavy():
    spec = W.WORKLOADS["minilm_heavy"]
    wl = W.make_workload(spec)
    rows = CC.lemma1_table(wl, spec.b_min, spec.n_max, spec.encoder.d_model)
    assert all(r["within_bound"] for r in rows)
    r2 = [r for r in rows if r["plan"] == "R2"]
    r1 = [r for r in rows if r["plan"] == "R1"]
    assert all(r["max_texts"] <= spec.n_max for r in r2)
    # without the cap a single oversized partition drives the largest call
    assert all(r["max_texts"] > 10 * spec.n_max for r in r1)


def test_lemma1_memory_worked_example(golden_dir):
    """M(S) = S L + 4 S d against the paper's worked example (Sec. 4.3):
    500K texts of 47 bytes with d = 384 hold 23.5 MB of text and 768 MB of
    embeddings, 791.5 MB in all; eq. (memory) rounds it to 791 MB."""
    g = json.load(open(os.path.join(golden_dir, "lemma1_memory.json")))
    S, L, d = g["S"], g["L_bytes"], g["d"]
    total = OP.superbatch_memory(S, L, d)
    assert total == pytest.approx(g["total_MB"] * 1e6, abs=0.5)
    assert OP.superbatch_memory(S, L, 0) == pytest.approx(g["text_MB"] * 1e6, abs=0.5)
    assert OP.superbatch_memory(S, 0, d) == pytest.approx(g["embeddings_MB"] * 1e6, abs=0.5)
    assert round(total / 1e6) == pytest.approx(g["eq_memory_MB_rounded"], abs=1)
    # int32 token IDs on the device: L = 4 bytes per token of the text
    assert OP.device_superbatch_memory(S, 12 * S, d) == OP.superbatch_memory(S, 48, d)
