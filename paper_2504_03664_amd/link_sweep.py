"""Chunk-size sweep of the host-to-device transfer (the paper's block-size
experiment, Appendix A, redone for this link): the rate of pinned-to-HBM
copies issued back to back in chunks of 1 MiB .. 512 MiB on one or two
copy streams, and the decode throughput of a workload as a function of
pipo_policy.chunk_bytes.  Prints one JSON line.

    python -m paper_2504_03664_amd.link_sweep [--workload I] [--steps K]
"""
from __future__ import annotations

import argparse
import json
import sys
import time

import numpy as np

from . import binding as B
from .model import Decoder, HostWeights

CHUNKS_MB = (1, 2, 4, 8, 16, 32, 64, 128, 256, 512)


def main() -> int:
    import synth
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, default=1, help="index into synth.WORKLOADS")
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--total-mb", type=int, default=2048)
    args = ap.parse_args()

    out = {"link": [], "decode": []}
    total = args.total_mb << 20
    for ns in (1, 2):
        for c in CHUNKS_MB:
            g = B.pipo_measure_h2d_chunked(total, c << 20, 5, ns)
            out["link"].append({"chunk_mb": c, "streams": ns, "gbps": round(g, 2)})
            print(f"link chunk {c} MiB x{ns}: {g:.1f} GB/s", file=sys.stderr, flush=True)

    wl = synth.WORKLOADS[args.workload]
    hw = HostWeights(wl.shape, wl.wfmt, synth.SyntheticOPT(wl.shape, seed=synth.DEFAULT_SEED,
                                                          wfmt=wl.wfmt))
    prompt = synth.prompt_tokens(wl.batch, wl.prompt, wl.shape.vocab, seed=1, stream=args.workload)
    try:
        for ns in (1, 2):
            for c in (1, 4, 16, 64, 256):
                with Decoder(hw, kv_on_host=wl.kv_on_host, kv_fmt=wl.kv_fmt, n_h2d_streams=ns,
                             chunk_bytes=c << 20, max_batch=wl.batch,
                             max_seq=wl.prompt + 2 + args.steps) as dec:
                    nxt, _ = dec.prefill(prompt)
                    nxt, _ = dec.decode(nxt)
                    dec.reset_stats()
                    t0 = time.perf_counter()
                    for _ in range(args.steps):
                        nxt, _ = dec.decode(nxt)
                    dt = time.perf_counter() - t0
                    st = dec.stats()
                tps = wl.batch * args.steps / dt
                out["decode"].append({"chunk_mb": c, "streams": ns, "tokens_per_s": round(tps, 2),
                                      "h2d_bytes_per_step": st["h2d_bytes"] // args.steps})
                print(f"decode chunk {c} MiB x{ns}: {tps:.2f} tokens/s", file=sys.stderr,
                      flush=True)
    finally:
        hw.free()
    out["workload"] = wl.name
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
