"""The trace-based GPU-busy figures (paper_2504_03664_amd/trace_busy.py) on
hand-made rocprofv3-style traces."""
import csv

import pytest

from paper_2504_03664_amd.trace_busy import analyse, union_length


def test_union_length_by_hand():
    iv = [(0, 10), (5, 15), (20, 30), (29, 31), (40, 41)]
    assert union_length(iv, 0, 100) == 15 + 11 + 1
    assert union_length(iv, 8, 25) == 7 + 5
    assert union_length([], 0, 10) == 0
    assert union_length([(0, 10)], 10, 20) == 0


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def test_analyse_window_and_fractions(tmp_path):
    # passes end at 100 (prefill), 200 (warm-up), 300, 400 (timed)
    k = []
    for e in (100, 200, 300, 400):
        k.append(["KERNEL_DISPATCH", "pipo::argmax_k(float const*)", e - 6, e - 3])
        k.append(["KERNEL_DISPATCH", "pipo::argmax_merge_k(float2 const*)", e - 2, e])
    k.append(["KERNEL_DISPATCH", "gemm", 210, 230])
    _write(tmp_path / "b_kernel_trace.csv", ["Kind", "Kernel_Name", "Start_Timestamp",
                                             "End_Timestamp"], k)
    c = [["MEMORY_COPY", "MEMORY_COPY_HOST_TO_DEVICE", 220, 290, 7000],
         ["MEMORY_COPY", "MEMORY_COPY_HOST_TO_DEVICE", 300, 380, 8000],
         ["MEMORY_COPY", "MEMORY_COPY_DEVICE_TO_HOST", 395, 399, 8],
         ["MEMORY_COPY", "MEMORY_COPY_HOST_TO_DEVICE", 50, 90, 1]]     # before the window
    _write(tmp_path / "b_memory_copy_trace.csv", ["Kind", "Direction", "Start_Timestamp",
                                                  "End_Timestamp", "Bytes"], c)
    r = analyse(str(tmp_path), warmup=1, steps=2)
    assert r["window_ms"] == pytest.approx(200 / 1e6)
    # kernels in (200, 400]: gemm 210-230, argmax 294-297 and 298-300, 394-397 and
    # 398-400 -> 20 + 5 + 5
    assert r["kernel_busy_frac"] == pytest.approx(30 / 200)
    # copies: 220-290, 300-380, 395-399 -> 70 + 80 + 4
    assert r["copy_busy_frac"] == pytest.approx(154 / 200)
    # union: 210-290 (80), 294-297 (3), 298-380 (82), 394-400 (6)
    assert r["busy_frac"] == pytest.approx(171 / 200)
    assert r["h2d_bytes"] == 15000
    with pytest.raises(ValueError):
        analyse(str(tmp_path), warmup=2, steps=2)
