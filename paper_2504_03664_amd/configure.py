"""Print the automatic configuration (pipo_configure; Section 3.5, Eq. (1))
of a workload for given memory budgets, with the cost of every placement
and pipeline it weighed.

    python -m paper_2504_03664_amd.configure --workload 3 --hbm-gb 24 [--host-gb 512]
"""
from __future__ import annotations

import argparse
import itertools
import json
import sys

from . import binding as B
from .model import c_policy, c_shape


def main() -> int:
    import synth
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, default=3, help="index into synth.WORKLOADS")
    ap.add_argument("--hbm-gb", type=float, default=0, help="0: the device's free memory")
    ap.add_argument("--host-gb", type=float, default=0, help="0: the system's available memory")
    args = ap.parse_args()
    wl = synth.WORKLOADS[args.workload]
    shape = c_shape(wl.shape)
    max_seq = wl.prompt + wl.gen
    wf = B.PIPO_W_FP16 if wl.wfmt == "fp16" else B.PIPO_W_INT4_G64
    kf = B.PIPO_KV_FP16 if wl.kv_fmt == "fp16" else B.PIPO_KV_INT4_G64
    options = []
    for w, e, k, n in itertools.product((0, 1), (0, 1), (0, 1), (3, 2, 1)):
        if k > w or (not w and not e and n != 3):
            continue
        p = B.pipo_plan_policy(shape, c_policy(wfmt=wl.wfmt, kv_fmt=wl.kv_fmt, max_batch=wl.batch,
                                               max_seq=max_seq, weights_on_host=bool(w),
                                               embed_on_host=bool(e), kv_on_host=bool(k),
                                               n_weight_slots=n))
        options.append({"weights_on_host": w, "embed_on_host": e, "kv_on_host": k,
                        "n_weight_slots": n, "hbm_gb": round(p["hbm_bytes"] / 1e9, 3),
                        "host_kv_gb": round(p["host_kv_bytes"] / 1e9, 3),
                        "h2d_gb_per_step": round(p["h2d_bytes_per_step"] / 1e9, 3)})
    out = {"workload": wl.name, "options": options}
    try:
        pol, plan = B.pipo_configure(shape, wf, kf, wl.batch, max_seq, int(args.hbm_gb * 1e9),
                                     int(args.host_gb * 1e9))
        out["chosen"] = {"weights_on_host": pol.weights_on_host,
                         "embed_on_host": pol.embed_on_host, "kv_on_host": pol.kv_on_host,
                         "n_weight_slots": pol.n_weight_slots,
                         "pipeline": ("performance-optimized"
                                      if plan["pipeline"] == B.PIPO_PIPE_PERFORMANCE
                                      else "memory-efficient"),
                         "hbm_budget_gb": round(pol.hbm_budget_bytes / 1e9, 3),
                         "plan": plan}
    except B.PipoError as e:
        out["chosen"] = None
        out["error"] = str(e)
    print(json.dumps(out, indent=1))
    return 0


if __name__ == "__main__":
    sys.exit(main())
