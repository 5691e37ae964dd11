"""A kernel of known HBM traffic, for calibrating rocprofv3 counters.

    rocprofv3 --pmc FETCH_SIZE -- python3 -m paper_2504_03664_amd.calibrate_copy

runs pipo_op_copy over `--mib` MiB (default 1024) `--iters` times: each
dispatch reads and writes exactly that many bytes, so FETCH_SIZE and
WRITE_SIZE per dispatch (KiB) divided by mib * 1024 give the counters'
scale factors.
"""
import argparse
import sys

from . import binding as B


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--mib", type=int, default=1024)
    ap.add_argument("--iters", type=int, default=5)
    a = ap.parse_args()
    n = a.mib << 20
    src, dst = B.DeviceBuffer(n), B.DeviceBuffer(n)
    for _ in range(a.iters):
        B.pipo_op_copy(dst.ptr, src.ptr, n)
    B.pipo_dev_synchronize()
    print(f"copied {a.mib} MiB x {a.iters}", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
