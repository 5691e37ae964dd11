"""GPU-busy fractions of a decode run from a rocprofv3 trace.

    rocprofv3 --kernel-trace --memory-copy-trace --output-format csv -d OUT -o bench \\
        -- python3 bench.py --runs 1 --no-timestamps --no-cpu-baseline ...
    python -m paper_2504_03664_amd.trace_busy OUT --warmup W --steps K

A pass (the prefill, or one decode step) ends with its argmax kernels, so
the end of the last argmax kernel of pass i marks the end of pass i; the
timed window of bench.py's single run is (end of pass W, end of pass W + K]:
after the prefill (pass 0) and the W warm-up steps.  Over that window the
script takes the union of the kernel intervals and of the memory-copy
intervals (the copy engines: host-to-device weight and KV loads,
device-to-host KV saves and token readbacks) and reports

* busy: |kernels U copies| / window,
* copy busy: |copies| / window (the pipeline's transfer bubbles show here),
* kernel busy: |kernels| / window,
* the host-to-device bytes inside the window and their rate, when the trace
  gives copy sizes.

These are the figures bench.py also derives from HIP events around every
operation (its gpu_busy object), here from the profiler's own timestamps and
over steps run without those events.
"""
from __future__ import annotations

import argparse
import csv
import glob
import os
import sys
from typing import List, Tuple

Interval = Tuple[int, int]


def _rows(path: str) -> List[dict]:
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _find(out_dir: str, suffix: str) -> str:
    hits = sorted(glob.glob(os.path.join(out_dir, "**", f"*{suffix}"), recursive=True))
    if not hits:
        raise FileNotFoundError(f"no *{suffix} under {out_dir}")
    return hits[0]


def union_length(iv: List[Interval], lo: int, hi: int) -> int:
    """Length of the union of intervals clipped to [lo, hi)."""
    clipped = sorted((max(a, lo), min(b, hi)) for a, b in iv if b > lo and a < hi)
    total, cur_a, cur_b = 0, None, None
    for a, b in clipped:
        if cur_b is None or a > cur_b:
            if cur_b is not None:
                total += cur_b - cur_a
            cur_a, cur_b = a, b
        else:
            cur_b = max(cur_b, b)
    if cur_b is not None:
        total += cur_b - cur_a
    return total


def pass_ends(kernels: List[dict]) -> List[int]:
    """End timestamp of every pass: its argmax merge kernel (or the
    single-pass argmax kernel where no merge kernel runs)."""
    merge = sorted(int(r["End_Timestamp"]) for r in kernels if "argmax_merge_k" in r["Kernel_Name"])
    if merge:
        return merge
    return sorted(int(r["End_Timestamp"]) for r in kernels if "argmax_k" in r["Kernel_Name"])


def _bytes_column(row: dict):
    for key in ("Bytes", "Size", "Copy_Bytes", "Copy_Size"):
        if key in row:
            return key
    return None


def analyse(out_dir: str, warmup: int, steps: int) -> dict:
    kernels = _rows(_find(out_dir, "kernel_trace.csv"))
    copies = _rows(_find(out_dir, "memory_copy_trace.csv"))
    ends = pass_ends(kernels)
    if len(ends) < 1 + warmup + steps:
        raise ValueError(f"{len(ends)} passes in the trace, fewer than 1 + {warmup} + {steps}")
    lo, hi = ends[warmup], ends[warmup + steps]
    kiv = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in kernels]
    civ = [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in copies]
    window = hi - lo
    res = {"window_ms": window / 1e6, "steps": steps,
           "busy_frac": union_length(kiv + civ, lo, hi) / window,
           "copy_busy_frac": union_length(civ, lo, hi) / window,
           "kernel_busy_frac": union_length(kiv, lo, hi) / window,
           "kernels_in_window": sum(1 for a, b in kiv if lo <= a < hi),
           "copies_in_window": sum(1 for a, b in civ if lo <= a < hi)}
    key = _bytes_column(copies[0]) if copies else None
    if key:
        h2d = [r for r in copies if "HOST_TO_DEVICE" in r.get("Direction", "").upper()
               and lo <= int(r["Start_Timestamp"]) < hi]
        nb = sum(int(r[key]) for r in h2d)
        res["h2d_bytes"] = nb
        res["h2d_gbps"] = nb / window          # bytes per ns = GB/s
        res["h2d_copy_busy_frac"] = union_length(
            [(int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in h2d], lo, hi) / window
    return res


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("out_dir")
    ap.add_argument("--warmup", type=int, required=True)
    ap.add_argument("--steps", type=int, required=True)
    a = ap.parse_args(argv)
    r = analyse(a.out_dir, a.warmup, a.steps)
    print(f"| figure | value |\n|---|---|")
    for k, v in r.items():
        print(f"| {k} | {v:.4f} |" if isinstance(v, float) else f"| {k} | {v} |")
    return 0


if __name__ == "__main__":
    sys.exit(main())
