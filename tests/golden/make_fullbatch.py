"""Write the oracle's teacher-forced results at the full workload batches.

For each case below this script runs the CPU oracle (``oracle/``) on the
seeded synthetic inputs of a workload (``synth/``) and stores, for every
batch row and every generated position, what a GPU run of the same inputs
is compared with in ``tests/test_gpu_fullbatch.py``:

* the 8 largest logits and their token ids (argmax agreement, and the
  near-tie check of every disagreement),
* the largest |logit| of the position (the scale of the normwise error),
* the logits of 64 fixed token ids drawn once per workload (a sampled normwise
  error at every position; rows 0 and b - 1 are also recomputed in full by
  the test itself).

Teacher forcing (the prompt, then gen - 1 seeded uniform ids) makes every
input independent of what either implementation generates, so these
values come from the oracle alone.  Nothing here imports the GPU library.

Readings: ``fp32`` is the plain fp32 decoder; ``fp16ops`` is the same with
every tensor the paper keeps in fp16 (activations, Section 4.1; expanded
INT4 weights) rounded to fp16 -- the precision in which the kernels take
their integer decisions (argmax, INT4 cache codes).

    python tests/golden/make_fullbatch.py            # every missing case
    python tests/golden/make_fullbatch.py NAME ...   # the named cases (rewritten)
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402
from oracle import decoder_for  # noqa: E402

OUT_DIR = os.path.join(HERE, "fullbatch")
TOP = 8
N_SAMPLED = 64

# name: workload index, layers (None = every layer), rows (None = the whole
# batch), oracle reading, INT4 cache entries, zero key/value projections
CASES = {
    # two-layer slices, whole batch
    "opt-6.7b-l2": dict(widx=1, layers=2),
    "opt-6.7b-l2-fp16ops": dict(widx=1, layers=2, reading="fp16ops"),
    "opt-13b-int4-l2": dict(widx=2, layers=2),
    "opt-30b-l2": dict(widx=3, layers=2),
    "opt-30b-int4-kvhost-l2": dict(widx=4, layers=2),
    "opt-30b-int4-kv4-l2-fp16ops": dict(widx=5, layers=2, reading="fp16ops"),
    "opt-30b-int4-kv4-l2-fp32": dict(widx=5, layers=2),
    "opt-30b-int4-kv4-zerokv-l2": dict(widx=5, layers=2, zero_kv=True),
    "llama3.1-8b-l2": dict(widx=6, layers=2),
    "llama3.1-8b-int4-l2": dict(widx=7, layers=2),
    # every layer, whole batch (or the first 16 rows at batch 64 / 128)
    "opt-6.7b-full": dict(widx=1),
    "opt-13b-int4-full": dict(widx=2),
    "llama3.1-8b-full": dict(widx=6),
    "llama3.1-8b-int4-full": dict(widx=7),
    "llama3.1-8b-int4-full-fp16ops": dict(widx=7, reading="fp16ops"),
    "opt-30b-full-r16": dict(widx=3, rows=16),
    "opt-30b-int4-kvhost-full-r16": dict(widx=4, rows=16),
}


def case_inputs(case: dict):
    """(workload, model provider, prompt [R][P], forced [R][gen-1], rows)."""
    wl = synth.WORKLOADS[case["widx"]]
    shape = wl.shape if case.get("layers") is None else wl.shape.with_layers(case["layers"])
    model = synth.synthetic_model(shape, seed=synth.DEFAULT_SEED, wfmt=wl.wfmt)
    if case.get("zero_kv"):
        model = synth.ZeroKV(model)
    prompt, forced = synth.teacher_tokens(wl, stream=case["widx"])
    rows = np.arange(wl.batch if case.get("rows") is None else case["rows"])
    return wl, shape, model, prompt[rows], forced[rows], rows


def sampled_ids(widx: int, vocab: int) -> np.ndarray:
    """The token ids whose logits are stored at every position (one set per
    workload, so the cases of a workload can be compared with each other)."""
    rng = np.random.Generator(np.random.Philox(key=np.array([widx, 0x53414D50], np.uint64)))
    return np.sort(rng.choice(vocab, size=N_SAMPLED, replace=False)).astype(np.int32)


def run_case(name: str, case: dict) -> str:
    wl, shape, model, prompt, forced, rows = case_inputs(case)
    reading = case.get("reading", "fp32")
    kv_int4 = wl.kv_fmt == "int4"
    dec = decoder_for(model, np.float32, kv_int4=kv_int4, fp16_operands=(reading == "fp16ops"))
    tokens = np.concatenate([prompt, forced], axis=1)
    t0 = time.time()
    R, G = len(rows), wl.gen
    samp = sampled_ids(case["widx"], shape.vocab)
    top_idx = np.empty((R, G, TOP), np.int32)
    top_val = np.empty((R, G, TOP), np.float32)
    absmax = np.empty((R, G), np.float32)
    samp_val = np.empty((R, G, N_SAMPLED), np.float32)
    S = tokens.shape[1]
    chunk = max(1, int(1e9 // (S * shape.d_model * 4)))     # ~1 GB of hidden states
    for c0 in range(0, R, chunk):
        lg = dec.forward(tokens[c0:c0 + chunk], last=G)           # [r][G][V] fp32
        part = np.argpartition(-lg, TOP, axis=-1)[..., :TOP]
        vals = np.take_along_axis(lg, part, axis=-1)
        # order: value descending, then token id ascending (ties to the lowest id)
        order = np.lexsort((part, -vals), axis=-1)
        top_idx[c0:c0 + chunk] = np.take_along_axis(part, order, axis=-1)
        top_val[c0:c0 + chunk] = np.take_along_axis(vals, order, axis=-1)
        absmax[c0:c0 + chunk] = np.abs(lg).max(axis=-1)
        samp_val[c0:c0 + chunk] = lg[..., samp]
        # the stored first entry is the oracle's greedy token
        assert np.array_equal(top_idx[c0:c0 + chunk, :, 0], lg.argmax(-1))
        print(f"  {name}: rows {c0}..{min(c0 + chunk, R) - 1} done "
              f"({time.time() - t0:.0f} s)", flush=True)
    meta = dict(case=name, workload=wl.name, layers=shape.n_layers, rows=R,
                reading=reading, kv_int4=kv_int4, zero_kv=bool(case.get("zero_kv")),
                prompt_seed=1, forced_seed=2, stream=case["widx"],
                weight_seed=synth.DEFAULT_SEED, seconds=round(time.time() - t0, 1),
                writer="tests/golden/make_fullbatch.py")
    os.makedirs(OUT_DIR, exist_ok=True)
    path = os.path.join(OUT_DIR, name + ".npz")
    np.savez_compressed(path, top_idx=top_idx, top_val=top_val, absmax=absmax,
                        samp_idx=samp, samp_val=samp_val, rows=rows.astype(np.int32),
                        meta=np.array(json.dumps(meta)))
    return path


def main(argv):
    names = argv or [n for n in CASES if not os.path.exists(os.path.join(OUT_DIR, n + ".npz"))]
    for n in names:
        print(f"{n}: {CASES[n]}", flush=True)
        print(f"  wrote {run_case(n, CASES[n])}", flush=True)


if __name__ == "__main__":
    main(sys.argv[1:])
