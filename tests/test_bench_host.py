"""Host logic of bench.py (no GPU): the one-GPU guard, and the rocprofv3 summaries.  The
summaries are the kernel table, the shader clock / MFMA occupancy, the GEMM and bandwidth-bound
kernel HBM traffic, and the digest check that nulls a stale traffic figure.  They are fed
synthetic counter CSVs whose answers are known."""
from __future__ import annotations

import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

GEMM = {0: "void rlk::(anonymous namespace)::k_gemm<rlk::bf16_t, 0, true, false>(rlk::GemmArgs)",
        1: "void rlk::(anonymous namespace)::k_gemm<rlk::bf16_t, 1, false, false>(rlk::GemmArgs)",
        2: "void rlk::(anonymous namespace)::k_gemm<rlk::bf16_t, 2, false, false>(rlk::GemmArgs)"}
COPY = "void at::native::vectorized_elementwise_kernel<4, at::native::neg_kernel_cuda(at::TensorIterator&)>"
DZ = "void rlk::(anonymous namespace)::k_dz<unsigned short, false>(rlk::DzParams)"

FIELDS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _write_counters(path, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_stats_summary_names_bf16_and_fp32_gemms(tmp_path):
    p = tmp_path / "stats.csv"
    with open(p, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Name", "Calls", "TotalDurationNs", "AverageNs", "MinNs", "MaxNs",
                                          "Percentage"])
        w.writeheader()
        w.writerow(dict(Name=GEMM[0], Calls=13, TotalDurationNs=13e6, AverageNs=1e6, MinNs=5e4, MaxNs=2e6,
                        Percentage=50.0))
        w.writerow(dict(Name="void rlk::(anonymous namespace)::k_gemm<float, 2, false, false>(rlk::GemmArgs)",
                        Calls=1, TotalDurationNs=1e3, AverageNs=1e3, MinNs=1e3, MaxNs=1e3, Percentage=1.0))
        w.writerow(dict(Name="some_other_kernel", Calls=1, TotalDurationNs=1, AverageNs=1, MinNs=1, MaxNs=1,
                        Percentage=0.0))
    out = bench.stats_summary(str(p), "title", "cmd")
    assert "k_gemm<bf16_t,fwd_lse,store_q=true,ktail=false>" in out
    assert "k_gemm<float,dw,store_q=false,ktail=false>" in out
    assert "some_other_kernel" not in out
    line = [l for l in out.splitlines() if "fwd_lse" in l][0].split()
    assert line[1] == "13" and float(line[3]) == 1000.0  # calls, average in microseconds


def test_occupancy_summary_recovers_clock_and_occupancy(tmp_path):
    # one 2 ms dh launch at 1.5 GHz with the MFMA pipe 60 % busy on every SIMD, and a short launch
    # (an empty chunk) that the summary must leave out
    ns = 2_000_000
    cyc = 1.5e9 * ns * 1e-9
    rows = []
    for did, dur in ((1, ns), (2, 50_000)):
        base = dict(Dispatch_Id=did, Kernel_Name=GEMM[1], Start_Timestamp=0, End_Timestamp=dur)
        rows += [dict(base, Counter_Name="GRBM_GUI_ACTIVE", Counter_Value=cyc * bench.N_XCD),
                 dict(base, Counter_Name="SQ_VALU_MFMA_BUSY_CYCLES", Counter_Value=0.6 * cyc * bench.N_SIMD),
                 dict(base, Counter_Name="SQ_WAVE_CYCLES", Counter_Value=1000.0),
                 dict(base, Counter_Name="SQ_WAIT_ANY", Counter_Value=250.0)]
    p = tmp_path / "occ.csv"
    _write_counters(p, rows)
    out = bench.occupancy_summary(str(p), "t", "c")
    line = [l for l in out.splitlines() if l.startswith("dh_gemm")][0].split()
    assert line[1] == "1"                       # the short launch is left out
    assert abs(float(line[3]) - 1.5) < 0.01     # GHz
    assert abs(float(line[4]) - 0.6) < 1e-3     # MFMA occupancy
    assert abs(float(line[5]) - 0.25) < 1e-3    # waiting fraction


def test_occupancy_summary_counts_executed_mfma_flops(tmp_path, monkeypatch):
    # SQ_INSTS_VALU_MFMA_MOPS_BF16 counts 512-FLOP units over every launch, short ones included
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    rows = []
    for did, (kind, mops, dur) in enumerate(((0, 1e9, 2_000_000), (1, 2e9, 3_000_000), (2, 3e9, 40_000))):
        base = dict(Dispatch_Id=did, Kernel_Name=GEMM[kind], Start_Timestamp=0, End_Timestamp=dur)
        rows += [dict(base, Counter_Name="GRBM_GUI_ACTIVE", Counter_Value=1e6 * bench.N_XCD),
                 dict(base, Counter_Name="SQ_VALU_MFMA_BUSY_CYCLES", Counter_Value=5e5 * bench.N_SIMD),
                 dict(base, Counter_Name="SQ_WAVE_CYCLES", Counter_Value=10.0),
                 dict(base, Counter_Name="SQ_WAIT_ANY", Counter_Value=1.0),
                 dict(base, Counter_Name="SQ_INSTS_VALU_MFMA_MOPS_BF16", Counter_Value=mops)]
    p = tmp_path / "occ.csv"
    _write_counters(p, rows)
    text = bench.occupancy_summary(str(p), "t", "c")
    (tmp_path / "gemm_occupancy_tiny_fp32.txt").write_text(text)
    flop, occ = bench.read_occupancy("tiny_fp32", bench.kernel_source_digest())
    assert flop == pytest.approx(6e9 * 512)
    assert occ["fwd_lse_gemm"] == pytest.approx(0.5) and "dw_gemm" not in occ   # the 40 us launch is left out
    assert bench.read_occupancy("tiny_fp32", "0" * 16) is None                     # other kernel sources


def test_host_policy_token_count_and_cpu_ranges():
    import numpy as np

    class St:
        cu_seqlens = np.array([0, 3, 5, 9])
        mask = np.array([1, 0, 1, 1, 1, 0, 1, 1, 0], np.uint8)
        group_ids = np.array([4, -1, 4])

    assert bench.host_policy_tokens(St) == 4
    assert bench.host_policy_tokens(St, exclusion=False) == 6
    assert bench._ranges([0, 1, 2, 3, 8, 10, 11]) == "0-3,8,10-11"


def _traffic_rows(counter, copy_kib, gemm_kib, dz_kib):
    rows = [dict(Dispatch_Id=1, Kernel_Name=COPY, Counter_Name=counter, Counter_Value=copy_kib,
                 Start_Timestamp=0, End_Timestamp=1)]
    for i, (kind, kib) in enumerate(gemm_kib.items()):
        for rep in range(2):
            rows.append(dict(Dispatch_Id=10 + 10 * i + rep, Kernel_Name=GEMM[kind], Counter_Name=counter,
                             Counter_Value=kib, Start_Timestamp=0, End_Timestamp=1))
    rows.append(dict(Dispatch_Id=99, Kernel_Name=DZ, Counter_Name=counter, Counter_Value=dz_kib,
                     Start_Timestamp=0, End_Timestamp=1))
    return rows


def test_traffic_summaries_scale_by_the_calibration_copy(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    # the fetch counter reports half of the copy's 1 MiB, the write counter all of it
    f, w = tmp_path / "f.csv", tmp_path / "w.csv"
    _write_counters(f, _traffic_rows("FETCH_SIZE", 512.0, {0: 100.0, 1: 200.0, 2: 300.0}, 1e6))
    _write_counters(w, _traffic_rows("WRITE_SIZE", 1024.0, {0: 10.0, 1: 20.0, 2: 30.0}, 5e5))
    paths = bench.traffic_summary(str(f), str(w), "tiny_fp32", 1, "fc", "wc")
    assert len(paths) == 3
    digest = bench.kernel_source_digest()
    # fwd: (100 * 2 + 10 * 1) KiB per launch
    assert bench.read_traffic("fwd_lse_gemm", "tiny_fp32", digest) == pytest.approx((200.0 + 10.0) * 1024)
    assert bench.read_traffic("dw_gemm", "tiny_fp32", digest) == pytest.approx((600.0 + 30.0) * 1024)
    # a summary taken from other kernel sources is not used
    assert bench.read_traffic("fwd_lse_gemm", "tiny_fp32", "0" * 16) is None
    hbm = bench.hbm_kernel_summary(str(f), str(w), "tiny_fp32", 1, "fc", "wc")
    line = [l for l in open(hbm) if l.startswith("k_dz")][0].split()
    assert float(line[2]) == pytest.approx((1e6 * 2 + 5e5) * 1024 / 1e9, rel=1e-3)


def test_traffic_summary_without_calibration_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--traffic-summary", "a.csv", "b.csv"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0 and "calibrate-copy-mib" in r.stderr
