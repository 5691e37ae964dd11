#!/usr/bin/env python3
"""Decode throughput of the pipelined-offloading decoder on one MI355X.

One step = one decode step of the whole batch: every layer's weights and the
output head stream from pinned host memory into rotating HBM slots while the
layers compute (and, for the KV-in-host workload, each layer's KV prefix
streams in and the new rows stream out).  Prints one JSON line on stdout;
progress goes to stderr.

    python bench.py [--steps K] [--warmup W] [--runs R] [--workload I]

Default workload: OPT-30B shape (48 layers, d 7168, 56 heads, FFN 28672),
fp16 weights, batch 64, prompt 512, 32 generated tokens, KV cache in HBM.
Each of R runs (default 3) is one whole generation: the prefill, W warm-up
decode steps, K timed decode steps (exactly K, bracketed by device
synchronisations), then untimed steps up to the workload's 32 tokens; the
reported throughput is the median run's, with the spread beside it.
--workload picks another entry of synth.WORKLOADS (OPT shapes, INT4 weights
and caches, the KV cache in host memory, LLaMA-3.1-8B shapes).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode tokens/s at 1 GPU; % of H2D-link roofline; GPU-busy %"
KERNEL_SOURCES = ("gemm.hip", "attention.hip", "device.h")
HBM_PEAK_GBPS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed decode steps (default 30; 4 for disk-tier workloads, whose "
                         "steps take seconds each)")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--runs", type=int, default=3,
                    help="timed generations (each: prefill, warm-up steps, timed steps, then "
                         "untimed steps up to the workload's generated length); the reported "
                         "throughput is their median")
    ap.add_argument("--workload", type=int, default=3,
                    help="index into synth.WORKLOADS (default: the OPT-30B fp16 decode)")
    ap.add_argument("--chunk-mb", type=int, default=64)
    ap.add_argument("--slots", type=int, default=3)
    ap.add_argument("--h2d-streams", type=int, default=2)
    ap.add_argument("--no-timestamps", action="store_true",
                    help="skip device timestamps (no busy %% or kernel roofline)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--segment-copies", action="store_true",
                    help="copy each tensor of a layer separately instead of one merged range "
                         "(ablation of the paper's data merging)")
    ap.add_argument("--layers", type=int, default=0, help="override layer count (testing only)")
    ap.add_argument("--disk-dir", default=None,
                    help="directory of the disk tier's file (disk workloads; default: the "
                         "system's temporary directory)")
    return ap.parse_args()


# the decode GEMM kernel plan of gemm.hip, restated to name the kernels in
# rocprofv3 output: (NF, KW, PD, KC) of the streaming kernel by (INT4, MF)
_STREAM_SEL = {(False, 2): (1, 8, 2, 128), (False, 4): (1, 8, 2, 128), (False, 8): (1, 8, 2, 128),
               (True, 2): (1, 8, 2, 256), (True, 4): (2, 8, 4, 256), (True, 8): (2, 8, 4, 128)}


def gemm_family(M):
    return "gemm_skinny" if M <= 16 else ("gemm_stream" if M <= 128 else "gemm_tiled")


def gemm_symbols(M, N, K, epi, w4, frag):
    """Kernel symbols one GEMM launches: skinny (M <= 16; 64 W rows per
    workgroup when N >= 12288), streaming (16 < M <= 128; K split into the
    largest power of two <= 8 keeping the grid within 256 workgroups, plus
    its combine kernel), tiled, or big tiles (at least 512 tiles of
    256 x 256); `frag`: W in fragment order."""
    b = "true" if w4 else "false"
    pk = "true" if frag else "false"
    if M <= 16:
        # (the SwiGLU epilogue, 5, always pairs two gate and two up fragments)
        nf = 4 if N >= 64 * 192 or epi == 5 else 1
        return [f"gemm_skinny<{nf}, 1, 8, 2, {b}, {epi}, {pk}>(GemmArgs)"]
    if -(-M // 256) * -(-N // 256) >= 512:
        return [f"gemm_big_w4<{epi}, {pk}>(GemmArgs)" if w4 else f"gemm_big_f16<{epi}, {pk}>(GemmArgs)"]
    if M > 128:
        return [f"gemm_tiled<{b}, {epi}, {pk}>(GemmArgs)"]
    mf = 2 if M <= 32 else (4 if M <= 64 else 8)
    nf, kw, pd, kc = _STREAM_SEL[(w4, mf)]
    if K % kc:
        pd, kc = (pd if kc == 128 else 2 * pd), 128
    blocks = -(-N // (16 * nf * kw))
    S = 1
    while S < 8 and blocks * 2 * S <= 256 and K % (2 * S * kc) == 0:
        S *= 2
    # fp16 grids left under 192 workgroups unsplit take 6 waves per workgroup
    if not w4 and kc == _STREAM_SEL[(w4, mf)][3] and S == 1 and blocks < 192 \
            and -(-N // (16 * nf * 6)) <= 256:
        kw = 6
    syms = [f"gemm_stream<{nf}, {mf}, {kw}, {pd}, {b}, {kc}, {epi}, {pk}>(GemmArgs, float*, long)"]
    if S > 1:
        # four columns per thread when N allows (the engine's partials are aligned)
        syms.append(f"gemm_combine<{epi}, {S}, {4 if N % 4 == 0 else 1}>(GemmArgs, float const*)")
    return syms


def profile_tag(workload_name):
    """Key of a workload's committed profile summaries: model and batch, plus
    where the KV cache lives and its format (a disk tier runs the kernels of
    the same workload and shares its key)."""
    toks = workload_name.split()
    return "_".join(toks[:2] + [t for t in toks[2:] if t in ("kv-host", "kv-int4")])


def measured_traffic(workload_name, symbols, optional=()):
    """HBM bytes per dispatch of the kernels `symbols` (summed, plus those of
    `optional` that the profile holds) from the committed rocprofv3 PMC
    summary of this workload, or None if there is none, a kernel of
    `symbols` is missing from it, or the kernel sources changed since it was
    taken.  Returns (bytes, summary path, the kernels counted)."""
    import hashlib
    tag = profile_tag(workload_name)
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{tag}.json")
    if not os.path.exists(path):
        return None, None, list(symbols)
    with open(path) as f:
        rec = json.load(f)
    h = hashlib.sha256()
    for src in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2504_03664_amd", "csrc", src), "rb") as f:
            h.update(f.read())
    if rec.get("kernel_source_sha256") != h.hexdigest():
        return None, None, list(symbols)
    if any(sym not in rec["per_dispatch"] for sym in symbols):
        return None, None, list(symbols)
    present = list(symbols) + [sym for sym in optional if sym in rec["per_dispatch"]]
    total = sum(rec["per_dispatch"][sym]["fetch_bytes"] + rec["per_dispatch"][sym]["write_bytes"]
                for sym in present)
    return total, os.path.relpath(path, ROOT).replace(".json", ".md"), present


def cpu_baseline(wl, seed, sample_layers=2, steps=3):
    """Time the CPU oracle on a bounded sample of the decode workload: `steps`
    decode steps of `sample_layers` layers at full batch and full context
    (KV prefix filled with synthetic values), plus the output head, scaled
    to all layers."""
    import synth
    from oracle import decoder_for
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas_threads = None
    shape = wl.shape.with_layers(sample_layers)
    gen = synth.synthetic_model(shape, seed=seed, wfmt=wl.wfmt)
    llama = getattr(shape, "family", "opt") == "llama"

    class Held:  # the sample's weights, drawn once (drawing is not the oracle's work)
        def __init__(self):
            self.shape, self.wfmt = gen.shape, gen.wfmt
            self._layers = [gen.layer(j) for j in range(sample_layers)]
            self._tok, self._lnf = gen.tok_emb(), gen.lnf()
            self._pos = None if llama else gen.pos_emb()
            self._head = gen.lm_head() if llama else None

        def layer(self, j):
            return self._layers[j]

        def tok_emb(self):
            return self._tok

        def pos_emb(self):
            return self._pos

        def lm_head(self):
            return self._head

        def lnf(self):
            return self._lnf

    held = Held()
    dec = decoder_for(held, np.float32, kv_int4=wl.kv_fmt == "int4")
    b, ctx = wl.batch, wl.prompt + 1
    rng = np.random.default_rng(0)
    d = shape.d_model
    dkv = shape.n_kv_heads * shape.head_dim if llama else d   # width of a cached row
    cache = [[(rng.standard_normal((ctx, dkv), dtype=np.float32),
               rng.standard_normal((ctx, dkv), dtype=np.float32)) for _ in range(b)]
             for _ in range(sample_layers)]
    toks = synth.prompt_tokens(b, 1, shape.vocab, seed=9)[:, 0]
    fresh = lambda: [[(k, v) for k, v in layer] for layer in cache]  # noqa: E731
    dec.decode(fresh(), toks)                                           # warm-up
    xs = [rng.standard_normal((1, d), dtype=np.float32) for _ in range(b)]
    t_dec = t_head = 0.0
    for _ in range(steps):
        c = fresh()
        t0 = time.perf_counter()
        dec.decode(c, toks)
        t1 = time.perf_counter()
        np.stack([dec.head(x)[0] for x in xs])
        t2 = time.perf_counter()
        t_dec += t1 - t0
        t_head += t2 - t1
    t_layers = max(t_dec - t_head, 0.0)
    per_step = (t_layers / steps) * wl.shape.n_layers / sample_layers + t_head / steps
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        cores = os.cpu_count()
    return {"value": b / per_step, "unit": "tokens/s",
            "cores": blas_threads or cores, "host_cores_visible": cores, "kind": "oracle",
            "sample": (f"{steps} decode steps of {sample_layers} of {wl.shape.n_layers} layers "
                       f"plus the output head, batch {b}, context {ctx} (synthetic KV prefix), "
                       f"fp32 numpy; layer time scaled by {wl.shape.n_layers}/{sample_layers}"),
            "seconds": t_layers + t_head}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this implementation runs on one GPU only (asked for {args.gpus}); the "
              "multi-GPU designs are described, not built", file=sys.stderr)
        return 2
    import synth
    from paper_2504_03664_amd import binding as B
    from paper_2504_03664_amd.model import Decoder, HostWeights

    wl = synth.WORKLOADS[args.workload]
    shape = wl.shape if args.layers <= 0 else wl.shape.with_layers(args.layers)
    W = args.warmup
    K = args.steps if args.steps is not None else (4 if wl.weights_on_disk else 30)
    R = max(1, args.runs if not wl.weights_on_disk else 1)
    # instrumented steps after the timed ones
    KI = 0 if args.no_timestamps else min(K, 2 if wl.weights_on_disk else 10)
    # each run generates the workload's tokens (more if W + K steps need more)
    gen = max(wl.gen, 1 + W + K)
    max_seq = wl.prompt + max(gen, 1 + W + K + KI)
    seed = synth.DEFAULT_SEED
    log(f"workload {wl.name}: {shape.n_layers} layers, d {shape.d_model}, batch {wl.batch}")

    t0 = time.time()
    hw = HostWeights(shape, wl.wfmt, synth.synthetic_model(shape, seed=seed, wfmt=wl.wfmt))
    log(f"weights drawn into pinned host memory in {time.time() - t0:.1f} s")

    peak1 = B.pipo_measure_h2d_peak(1 << 30, 10, 1)
    peak2 = B.pipo_measure_h2d_peak(1 << 30, 10, 2)
    peak = max(peak1, peak2)
    log(f"H2D link peak: {peak1:.1f} GB/s (1 stream), {peak2:.1f} GB/s (2 streams)")

    disk = None
    if wl.weights_on_disk:
        import tempfile
        disk = {"dir": args.disk_dir or tempfile.gettempdir()}
        t0 = time.time()
    dec = Decoder(hw, weights_on_host=True, embed_on_host=True, kv_on_host=wl.kv_on_host,
                  kv_fmt=wl.kv_fmt, weights_on_disk=wl.weights_on_disk,
                  disk_dir=disk["dir"] if disk else None,
                  n_weight_slots=args.slots, n_h2d_streams=args.h2d_streams,
                  chunk_bytes=args.chunk_mb << 20, max_batch=wl.batch, max_seq=max_seq,
                  debug_flags=B.PIPO_DBG_SEGMENT_COPIES if args.segment_copies else 0)
    if disk:
        log(f"disk tier file written in {time.time() - t0:.1f} s")
        # the disk's read rate: the tier's whole file (what a step reads) read
        # once the way decode reads it; for context also the best of 3 passes
        # over its first 16 GiB; and whether direct I/O is possible there
        dpeak = B.pipo_measure_disk_tier(dec.ctx, 1 << 50, 1)
        log(f"disk-tier file read at {dpeak:.2f} GB/s")
        dprefix = B.pipo_measure_disk_tier(dec.ctx, 16 << 30, 3)
        _, direct = B.pipo_measure_disk_read(disk["dir"], 64 << 20, args.chunk_mb << 20, 8, 1)
        log(f"disk-tier read rate in {disk['dir']}: {dpeak:.2f} GB/s over the file, "
            f"{dprefix:.2f} GB/s best over its first 16 GiB (direct I/O: {direct})")
        disk.update(peak_gbps=dpeak, prefix_gbps=dprefix, direct_io=direct)
    prompt = synth.prompt_tokens(wl.batch, wl.prompt, shape.vocab, seed=1, stream=args.workload)
    runs = []
    for run in range(R):
        # one generation: prefill, W warm-up steps, K timed steps, then the
        # rest of the workload's generation untimed (the last run's rest is
        # replaced by the instrumented steps)
        t0 = time.perf_counter()
        nxt, _ = dec.prefill(prompt)
        ttft_ms = (time.perf_counter() - t0) * 1e3
        log(f"run {run}: prefill {wl.batch}x{wl.prompt}: {ttft_ms:.0f} ms")
        for _ in range(W):
            nxt, _ = dec.decode(nxt)
        dec.reset_stats()
        step_s = []
        B.pipo_dev_synchronize()      # every stream idle: no load of a timed step runs early
        t0 = time.perf_counter()
        for i in range(K):
            ts = time.perf_counter()
            nxt, _ = dec.decode(nxt)
            step_s.append(time.perf_counter() - ts)
            if step_s[-1] > 2.0:   # slow (disk-tier) steps: a progress line each
                log(f"decode step {i}: {step_s[-1]:.2f} s")
        B.pipo_dev_synchronize()      # and the loads the last step started ahead are done
        dt = time.perf_counter() - t0
        st = dec.stats()
        log(f"run {run}: {K} decode steps in {dt:.3f} s ({wl.batch * K / dt:.3f} tokens/s)")
        runs.append(dict(dt=dt, st=st, step_s=step_s, ttft_ms=ttft_ms))
        if run + 1 < R:
            for _ in range(gen - 1 - W - K):
                nxt, _ = dec.decode(nxt)
    # the median run (by throughput) is the one reported
    order = sorted(range(R), key=lambda i: runs[i]["dt"])
    med = runs[order[R // 2]]
    dt, st, step_s, ttft_ms = med["dt"], med["st"], med["step_s"], med["ttft_ms"]
    run_values = [wl.batch * K / r["dt"] for r in runs]
    if KI:
        # device timestamps around every copy and kernel, over separate
        # steps: they add events and a stream synchronisation per step, so
        # the throughput above is measured without them
        dec.set_timestamps(True)
        dec.reset_stats()
        ti = time.perf_counter()
        for i in range(KI):
            ts = time.perf_counter()
            nxt, _ = dec.decode(nxt)
            if time.perf_counter() - ts > 2.0:
                log(f"instrumented decode step {i}: {time.perf_counter() - ts:.2f} s")
        dti = time.perf_counter() - ti
        sti = dec.stats()
        log(f"{KI} instrumented decode steps in {dti:.3f} s")
    dec.close()

    value = wl.batch * K / dt
    bytes_step = st["h2d_bytes"] / K
    roof = wl.batch * peak * 1e9 / bytes_step
    sustained = st["h2d_bytes"] / dt / 1e9
    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "tokens/s", "n_gpus": 1,
        "steps": K, "warmup": W, "ms_per_step": round(dt / K * 1e3, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "fp16",
        "data": "synthetic",
        "config": {"workload": wl.name, "layers": shape.n_layers, "d_model": shape.d_model,
                   "batch": wl.batch, "prompt": wl.prompt,
                   "generated": gen, "warmup_steps": W, "timed_steps": K, "runs": R,
                   "weights": f"{wl.wfmt}, " + ("layers in the disk tier's file (disk -> pinned "
                                                "-> HBM), head pinned host" if wl.weights_on_disk
                                                else "pinned host") + ", streamed",
                   "kv_cache": ("host (pinned, or pageable through pinned staging), streamed"
                                if wl.kv_on_host else "HBM") + f", {wl.kv_fmt}",
                   "chunk_bytes": args.chunk_mb << 20, "slots": args.slots,
                   "h2d_streams": args.h2d_streams,
                   "copies": "per tensor" if args.segment_copies else "merged per layer"},
        "h2d_link": {"peak_gbps": round(peak, 2), "peak_1stream_gbps": round(peak1, 2),
                     "sustained_gbps": round(sustained, 2),
                     "frac_of_peak": round(sustained / peak, 4),
                     "bytes_per_step": int(bytes_step),
                     "staged_bytes_per_step": int(st["staged_bytes"] / K),
                     "roofline_tokens_per_s": round(roof, 3),
                     "frac_of_roofline": round(value / roof, 4)},
        "runs": {"n": R, "median": round(float(np.median(run_values)), 3),
                 "min": round(min(run_values), 3), "max": round(max(run_values), 3),
                 "spread_frac": round((max(run_values) - min(run_values))
                                      / float(np.median(run_values)), 4),
                 "tokens_per_s": [round(v, 3) for v in run_values],
                 "ttft_ms": [round(r["ttft_ms"], 1) for r in runs],
                 "source": "each run one whole generation (prefill, warm-up, timed and "
                           "untimed steps); value is the median run's"},
        "ttft_ms": round(float(np.median([r["ttft_ms"] for r in runs])), 1),
        **({"disk": {"peak_gbps": round(disk["peak_gbps"], 2),
                     "prefix_16gib_gbps": round(disk["prefix_gbps"], 2),
                     "direct_io": disk["direct_io"],
                     "bytes_per_step": int(st["disk_read_bytes"] / K),
                     "sustained_gbps": round(st["disk_read_bytes"] / dt / 1e9, 2),
                     "frac_of_peak": round(st["disk_read_bytes"] / dt / 1e9 / disk["peak_gbps"], 4),
                     "read_ms_per_step": round(st["disk_read_ms"] / K, 1),
                     "roofline_tokens_per_s": round(
                         wl.batch * disk["peak_gbps"] * 1e9 / (st["disk_read_bytes"] / K), 3),
                     "frac_of_roofline": round(
                         value / (wl.batch * disk["peak_gbps"] * 1e9 / (st["disk_read_bytes"] / K)),
                         4)}}
           if disk else {}),
        "step_ms": {"median": round(float(np.median(step_s)) * 1e3, 3),
                    "min": round(min(step_s) * 1e3, 3), "max": round(max(step_s) * 1e3, 3),
                    "source": "host clock around each pipo_decode_step (returns after the "
                              "token readback; later steps' loads may already run ahead)"},
    }
    if KI and sti["window_ms"] > 0:
        st = sti
        out["gpu_busy"] = {"busy_frac": round(st["busy_ms"] / st["window_ms"], 4),
                           "copy_busy_frac": round(st["copy_busy_ms"] / st["window_ms"], 4),
                           "kernel_busy_frac": round(st["kernel_busy_ms"] / st["window_ms"], 4),
                           "window_ms": round(st["window_ms"], 2),
                           "steps": KI,
                           "instrumented_tokens_per_s": round(wl.batch * KI / dti, 3),
                           "source": "HIP events around every copy and kernel, over "
                                     f"{KI} decode steps after the timed ones"}
        # dominant decode kernel, grouped by kernel symbol: the GEMM epilogue is
        # a template parameter, so the out-projection and FC2 share one symbol
        gemm = gemm_family(wl.batch)
        llama = getattr(shape, "family", "opt") == "llama"
        # LLaMA: FC1 is the gate/up GEMM (fp16 out) followed by the SwiGLU kernel,
        # QKV is followed by the rotary kernel
        # (at batch <= 16 the SwiGLU gate runs in the GEMM's epilogue)
        fc1_label = ((f"{gemm}<swiglu> (fc1)" if wl.batch <= 16 else f"{gemm}<f16>+swiglu (fc1)")
                     if llama else f"{gemm}<relu_f16> (fc1)")
        qkv_label = f"{gemm}<qkv>+rope (qkv)" if llama else f"{gemm}<qkv> (qkv)"
        families = {f"{gemm}<add_f32> (oproj+fc2)": ("oproj_decode", "fc2_decode"),
                    fc1_label: ("fc1_decode",),
                    qkv_label: ("qkv_decode",),
                    f"{gemm}<f32> (head)": ("head_decode",),
                    "attn_decode_k+combine (attention)": ("attn_decode",)}
        fam = {}
        for fname, members in families.items():
            ks = [st["kernels"][m] for m in members if m in st["kernels"]]
            if ks:
                fam[fname] = {k: sum(x[k] for x in ks) for k in ("launches", "total_ms",
                                                                  "alg_bytes", "alg_flops")}
        name, ks = max(fam.items(), key=lambda kv: kv[1]["total_ms"])
        avg_ms = ks["total_ms"] / ks["launches"]
        # the kernel's own roofline: HBM unless its arithmetic intensity
        # (algorithmic flops per algorithmic byte) exceeds the machine balance
        # of the fp16 MFMA peak over the HBM peak
        mfma_bound = ks["alg_flops"] > ks["alg_bytes"] * MFMA_F16_PEAK_TFLOPS / (HBM_PEAK_GBPS / 1e3)
        if mfma_bound:
            ach = ks["alg_flops"] / (ks["total_ms"] * 1e-3) / 1e12
            peak, unit = MFMA_F16_PEAK_TFLOPS, "TFLOP/s"
        else:
            ach = ks["alg_bytes"] / (ks["total_ms"] * 1e-3) / 1e9
            peak, unit = HBM_PEAK_GBPS, "GB/s"
        epi = {"oproj": 2, "fc1": (5 if wl.batch <= 16 else 0) if llama else 1, "qkv": 4, "head": 3}
        fam_key = name.split("(")[1].split("+")[0].rstrip(")")
        symbols, symbols_opt = None, []
        d, F, dh = shape.d_model, shape.d_ffn, shape.d_model // shape.n_heads
        hkv = shape.n_kv_heads if llama else shape.n_heads
        if fam_key in epi:
            nk = {"oproj": (d, d), "fc1": (2 * F if llama else F, d),
                  "qkv": (d + 2 * hkv * dh, d), "head": (shape.vocab, d)}
            # layer matrices stream in fragment order (HostWeights' default),
            # the output head is row-major
            symbols = gemm_symbols(wl.batch, *nk[fam_key], epi[fam_key],
                                   wl.wfmt == "int4" and fam_key != "head", fam_key != "head")
        elif fam_key == "attention":
            kv4 = "true" if wl.kv_fmt == "int4" else "false"
            G = shape.n_heads // hkv
            hp = 1 if G > 1 else (4 if hkv % 4 == 0 else (2 if hkv % 2 == 0 else 1))
            # fp16 rows: the library narrows workgroups to fewer heads while
            # that leaves fewer than 1536 of them
            while kv4 == "false" and hp > 1 and wl.batch * (hkv // hp) < 1536:
                hp //= 2
            symbols = ([f"attn_decode_kv4_k<{dh}, {hp}>"] if kv4 == "true" and G == 1
                       else [f"attn_decode_k<{dh}, {G}, {hp}, {kv4}>"])
            # with key splits the launch also runs the merge kernel (one
            # dispatch per attention launch), whose bytes count too
            symbols_opt = [f"attn_decode_combine<{dh}>"]
        traffic, tsrc, counted = (measured_traffic(wl.name, symbols, symbols_opt) if symbols
                                  else (None, None, None))
        symbol = " + ".join(counted) if counted else None
        out["roofline"] = {"kernel": name, "symbol": symbol,
                           "bound": "mfma" if mfma_bound else "hbm",
                           "achieved": round(ach, 1), "peak": peak, "unit": unit,
                           "frac": round(ach / peak, 4),
                           "intensity_flop_per_byte": round(ks["alg_flops"] / ks["alg_bytes"], 2),
                           "launches": ks["launches"], "avg_launch_us": round(avg_ms * 1e3, 2),
                           "alg_bytes_per_launch": int(ks["alg_bytes"] / ks["launches"]),
                           "traffic": int(traffic) if traffic else None,
                           "traffic_source": tsrc}
        out["kernels"] = {k: {"launches": v["launches"],
                              "avg_us": round(v["total_ms"] / v["launches"] * 1e3, 2),
                              "gbps": round(v["alg_bytes"] / v["total_ms"] / 1e6, 1)}
                          for k, v in st["kernels"].items()}
    hw.free()
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(wl, seed)
        log(f"oracle: {out['cpu_baseline']['value']:.3f} tokens/s")
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
