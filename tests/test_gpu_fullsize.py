"""Checks at the full workload sizes that need no stored oracle results: a
whole row recomputed by the oracle over the whole vocabulary at full depth,
and a property that holds at any size (a row decoded in the full batch
matches the same row decoded alone).  The stored-result comparisons over
whole batches are in test_gpu_fullbatch.py."""
import numpy as np
import pytest

import synth
from oracle import decoder_for
from paper_2504_03664_amd.model import Decoder, HostWeights

pytestmark = pytest.mark.gpu

REL_TOL = 2e-2


def log(msg):
    print(msg, flush=True)


def normwise(g, o):
    return np.abs(g - o).max(axis=-1) / np.abs(o).max(axis=-1)


def test_opt67b_full_depth_rows_in_full():
    """OPT-6.7B shape (32 layers, batch 16, prompt 512, 32 tokens, weights
    streamed): rows 0 and 15 recomputed by the fp32 oracle over all 50272
    logits at every position."""
    wl = synth.WORKLOADS[1]
    log(f"{wl.name}: drawing weights")
    model = synth.SyntheticOPT(wl.shape, seed=synth.DEFAULT_SEED)
    prompt, forced = synth.teacher_tokens(wl, stream=1)
    hw = HostWeights(wl.shape, "fp16", model)
    try:
        log("  GPU generation")
        with Decoder(hw, max_batch=wl.batch, max_seq=wl.prompt + wl.gen,
                     chunk_bytes=64 << 20) as dec:
            toks, logits = dec.generate(prompt, wl.gen, want_logits=True, forced=forced)
    finally:
        hw.free()
    logits = np.stack(logits, axis=1)
    rows = [0, wl.batch - 1]
    log(f"  oracle on rows {rows}")
    ref = decoder_for(model, np.float32).forward(
        np.concatenate([prompt[rows], forced[rows]], axis=1), last=wl.gen)
    worst = max(float(normwise(logits[r].astype(np.float64), ref[i].astype(np.float64)).max())
                for i, r in enumerate(rows))
    log(f"  max normwise error {worst:.3e}")
    assert worst <= REL_TOL


def test_opt67b_rows_independent_of_batch():
    """Every row of the full batch-16 run matches the same row run alone
    (different GEMM variants, so equal up to rounding)."""
    wl = synth.WORKLOADS[1]
    shape = wl.shape.with_layers(8)
    model = synth.SyntheticOPT(shape, seed=synth.DEFAULT_SEED)
    hw = HostWeights(shape, "fp16", model)
    try:
        prompt = synth.prompt_tokens(wl.batch, wl.prompt, shape.vocab, seed=1, stream=1)
        log("batch-16 run (8 layers)")
        forced = synth.prompt_tokens(wl.batch, 7, shape.vocab, seed=2, stream=1)
        with Decoder(hw, max_batch=wl.batch, max_seq=wl.prompt + 8, chunk_bytes=64 << 20) as dec:
            toks, logits = dec.generate(prompt, 8, want_logits=True, forced=forced)
        logits = np.stack(logits, axis=1)
        for r in (1, 7, 15):
            log(f"  row {r} alone")
            with Decoder(hw, max_batch=1, max_seq=wl.prompt + 8, chunk_bytes=64 << 20) as dec:
                t1, l1 = dec.generate(prompt[r:r + 1], 8, want_logits=True,
                                      forced=forced[r:r + 1])
            l1 = np.stack(l1, axis=1)[0].astype(np.float64)
            e = normwise(logits[r].astype(np.float64), l1)
            assert e.max() <= 5e-3, (r, e.max())
    finally:
        hw.free()
