"""Host logic of the measurement helpers (no GPU): kernel classification of
rocprofv3 names, the copy-calibrated traffic arithmetic, the source-hash
gate on stored traffic figures, the MFMA-busy share, the roofline summary,
and bench.py's refusal of more than one GPU."""
import csv
import json
import os

import pytest

import bench
from paper_2605_01060_amd import profiling as P

LIN = "void surge::(anonymous namespace)::linear_bf16_kernel<256, 256, 64, 4, 2, {epi}, {order}>(x)"
ATTN = "void surge::(anonymous namespace)::attention_varlen_kernel<64>(x)"
COPY = "__amd_rocclr_copyBuffer"


def test_kernel_classification():
    assert P._epi(LIN.format(epi=4, order=1)) == 4
    assert P._epi(ATTN) == -1
    assert P.name_class(LIN.format(epi=0, order=0)) == "qkv"
    assert P.name_class(LIN.format(epi=3, order=0)) == "qkv"
    assert P.name_class(LIN.format(epi=4, order=1)) == "ffn1"
    for epi in (2, 5, 6):
        assert P.name_class(LIN.format(epi=epi, order=0)) == "residual"
    assert P.name_class(ATTN) == "attn"
    assert P.name_class("void surge::(anonymous namespace)::ln_rows_kernel<16>(x)") == "layernorm"
    assert P.name_class(COPY) is None


def test_residual_gemms_told_apart_by_dispatch_order():
    """The O-projection and FFN2 share one kernel instance: the one after
    FFN1 is FFN2, the one after QKV and attention is the O-projection."""
    qkv0, qkv = LIN.format(epi=0, order=0), LIN.format(epi=3, order=0)
    o0, res = LIN.format(epi=5, order=0), LIN.format(epi=6, order=0)
    ffn1 = LIN.format(epi=4, order=1)
    names = [COPY, "embed_ln_kernel", qkv0, ATTN, o0, ffn1, res,
             qkv, ATTN, res, ffn1, res, "pool_l2_kernel"]
    assert P.dispatch_classes(names) == [
        None, None, "qkv", "attn", "oproj", "ffn1", "ffn2",
        "qkv", "attn", "oproj", "ffn1", "ffn2", None]


def _counter_csv(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i, (name, value) in enumerate(rows):
            w.writerow([i, name, counter, value])


def test_traffic_scales_by_the_calibration_copy(tmp_path):
    copy_mib = 2048
    # the copy reads half of its bytes through FETCH_SIZE (scale 2) and all of
    # them through WRITE_SIZE (scale 1); smaller copies are not the calibration
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    ffn1 = LIN.format(epi=4, order=1)
    _counter_csv(fetch, "FETCH_SIZE", [(COPY, 1024.0), (COPY, copy_mib * 512.0),
                                       (ffn1, 1000.0), (ffn1, 3000.0), (ATTN, 7.0)])
    _counter_csv(write, "WRITE_SIZE", [(COPY, copy_mib * 1024.0), (ffn1, 500.0),
                                       (ffn1, 700.0)])
    rec = P.traffic(str(fetch), str(write), "ffn1", copy_mib)
    assert rec["fetch_scale"] == pytest.approx(2.0)
    assert rec["write_scale"] == pytest.approx(1.0)
    assert rec["fetch_dispatches"] == 2 and rec["write_dispatches"] == 2
    assert rec["fetch_bytes_per_launch"] == pytest.approx(2000.0 * 1024 * 2.0)
    assert rec["write_bytes_per_launch"] == pytest.approx(600.0 * 1024 * 1.0)
    assert rec["bytes_per_launch"] == pytest.approx(2000.0 * 2048 + 600.0 * 1024)
    assert rec["source_sha256"] == P.source_hash("ffn1")
    _counter_csv(fetch, "FETCH_SIZE", [(ffn1, 1.0)])
    with pytest.raises(SystemExit):  # no calibration copy in the run
        P.traffic(str(fetch), str(write), "ffn1", copy_mib)


def _traffic_md(root, cls, sha, value):
    os.makedirs(root / "profiles", exist_ok=True)
    rec = {"kernel_class": cls, "source_sha256": sha, "bytes_per_launch": value}
    (root / "profiles" / f"traffic_{cls}_bge.md").write_text(
        "header\n\n```json\n" + json.dumps(rec) + "\n```\n")


def test_stored_traffic_is_dropped_once_the_source_changes(tmp_path, monkeypatch):
    monkeypatch.setattr(P, "ROOT", str(tmp_path))
    assert P.load_traffic("attn", "bge") is None  # absent
    _traffic_md(tmp_path, "attn", P.source_hash("attn"), 1.5e9)
    assert P.load_traffic("attn", "bge") == pytest.approx(1.5e9)
    _traffic_md(tmp_path, "attn", "0" * 64, 1.5e9)  # taken on another source
    assert P.load_traffic("attn", "bge") is None


def test_mfma_busy_share(tmp_path):
    path = tmp_path / "mfma.csv"
    ffn1 = LIN.format(epi=4, order=1)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for d, (mfma, busy) in enumerate([(400.0, 200.0), (200.0, 100.0)]):
            w.writerow([d, ffn1, "SQ_VALU_MFMA_BUSY_CYCLES", mfma])
            w.writerow([d, ffn1, "SQ_BUSY_CU_CYCLES", busy])
        w.writerow([9, ATTN, "SQ_VALU_MFMA_BUSY_CYCLES", 1.0])  # incomplete pair
    res = P.mfma_busy(str(path))
    assert res["ffn1"]["dispatches"] == 2
    assert res["ffn1"]["mfma_busy_pct"] == pytest.approx(100.0 * 600.0 / (4 * 300.0))
    assert "attn" not in res


def test_roofline_summary_reads_one_profiled_step(tmp_path, monkeypatch):
    monkeypatch.setattr(P, "ROOT", str(tmp_path))  # no stored traffic
    line = {"value": 1000.0, "ms_per_step": 2000.0, "mfma_util_pct": 30.0, "steps": 3,
            "kernels_from": "one untimed step",
            "kernels": {"ffn1": {"launches": 492, "total_ms_per_step": 700.0, "avg_ms": 1.4,
                                 "tflops": 850.0, "gbs": 1400.0}},
            "roofline": {"kernel": "ffn1", "achieved": 845.0, "peak": 2516.6,
                         "unit": "TFLOP/s", "frac": 845.0 / 2516.6, "avg_launch_ms": 1.48}}
    path = tmp_path / "bench.json"
    path.write_text(json.dumps(line))
    md = P.roofline_markdown(str(path), "bge", "python bench.py")
    row = [l for l in md.splitlines() if l.startswith("| ffn1 ")][0]
    assert row.split("|")[2].strip() == "492"  # launches of the one step
    assert "frac 0.336" in md
    assert f"{100 * 850.0 / 2516.6:.1f}" in row


def test_bench_refuses_more_than_one_gpu(capsys):
    assert bench.main(["--gpus", "2"]) == 2
    out = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    assert "one GPU" in out["error"]


def test_clock_per_kernel_class(tmp_path):
    """GRBM_GUI_ACTIVE is summed over the 8 XCDs: clock = value / 8 /
    duration; the MFMA peak scales with it."""
    path = tmp_path / "clock.csv"
    ffn1 = LIN.format(epi=4, order=1)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                    "Start_Timestamp", "End_Timestamp"])
        w.writerow([0, ffn1, "GRBM_GUI_ACTIVE", 8 * 2.0 * 1000.0, 5000, 6000])  # 2.0 GHz, 1 us
        w.writerow([1, ffn1, "GRBM_GUI_ACTIVE", 8 * 2.2 * 3000.0, 7000, 10000])  # 2.2 GHz, 3 us
        w.writerow([1, ffn1, "SQ_BUSY_CYCLES", 123.0, 7000, 10000])  # other counters ignored
    res = P.clock(str(path))
    assert res["ffn1"]["dispatches"] == 2
    assert res["ffn1"]["ghz"] == pytest.approx((2.0 * 1000 + 2.2 * 3000) / 4000)
    assert res["ffn1"]["peak_at_clock_tflops"] == pytest.approx(2516.6 * res["ffn1"]["ghz"] / 2.4)
    assert res["ffn1"]["mean_us"] == pytest.approx(2.0)


def test_roofline_bound_follows_arithmetic_intensity(tmp_path, monkeypatch):
    """A kernel below the ridge (315 FLOP/B) is held to the HBM roof, one
    above it to the MFMA roof."""
    monkeypatch.setattr(P, "ROOT", str(tmp_path))
    line = {"value": 1.0, "ms_per_step": 100.0, "mfma_util_pct": 20.0, "steps": 1,
            "kernels": {"oproj": {"launches": 10, "total_ms_per_step": 10.0, "avg_ms": 1.0,
                                  "tflops": 500.0, "gbs": 4000.0},  # 125 FLOP/B
                        "ffn2": {"launches": 10, "total_ms_per_step": 20.0, "avg_ms": 2.0,
                                 "tflops": 1000.0, "gbs": 2000.0}}}  # 500 FLOP/B
    path = tmp_path / "bench.json"
    path.write_text(json.dumps(line))
    md = P.roofline_markdown(str(path), "minilm", "python bench.py --workload minilm")
    oproj = [l for l in md.splitlines() if l.startswith("| oproj ")][0].split("|")
    ffn2 = [l for l in md.splitlines() if l.startswith("| ffn2 ")][0].split("|")
    assert oproj[7].strip() == "hbm" and oproj[9].strip() == f"{100 * 4000 / 8000:.1f}"
    assert ffn2[7].strip() == "mfma" and ffn2[9].strip() == f"{100 * 1000 / 2516.6:.1f}"


def test_traffic_of_the_two_residual_gemms(tmp_path):
    """Counters of O-projection and FFN2 dispatches (one kernel instance)
    land in their own classes."""
    fetch = tmp_path / "fetch.csv"
    write = tmp_path / "write.csv"
    qkv, res, ffn1 = (LIN.format(epi=3, order=0), LIN.format(epi=6, order=0),
                      LIN.format(epi=4, order=1))
    seq = [(COPY, 1024.0), (qkv, 1.0), (ATTN, 1.0), (res, 100.0), (ffn1, 1.0), (res, 300.0),
           (qkv, 1.0), (ATTN, 1.0), (res, 120.0), (ffn1, 1.0), (res, 340.0)]
    _counter_csv(fetch, "FETCH_SIZE", seq)
    _counter_csv(write, "WRITE_SIZE", seq)
    o = P.traffic(str(fetch), str(write), "oproj", 1.0)
    f = P.traffic(str(fetch), str(write), "ffn2", 1.0)
    assert o["fetch_dispatches"] == f["fetch_dispatches"] == 2
    assert o["fetch_kib_per_dispatch_raw"] == pytest.approx(110.0)
    assert f["fetch_kib_per_dispatch_raw"] == pytest.approx(320.0)
    assert o["source_sha256"] == f["source_sha256"] == P.source_hash("ffn1")


def test_fabric_reads_count_each_request_at_its_size(tmp_path):
    path = tmp_path / "fabric.csv"
    ffn1 = LIN.format(epi=4, order=1)
    with open(path, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for d, n128 in enumerate([1000.0, 3000.0]):
            w.writerow([d, ffn1, "TCC_EA0_RDREQ_128B_sum", n128])
            w.writerow([d, ffn1, "TCC_EA0_RDREQ_64B_sum", 10.0])
            w.writerow([d, ffn1, "TCC_EA0_RDREQ_32B_sum", 2.0])
            w.writerow([d, ffn1, "TCC_EA0_RDREQ_sum", n128 + 12.0])
    res = P.fabric_reads(str(path))
    assert res["ffn1"]["dispatches"] == 2
    assert res["ffn1"]["read_bytes_per_launch"] == pytest.approx(2000.0 * 128 + 640 + 64)
    assert res["ffn1"]["accounted"] == pytest.approx(1.0)
