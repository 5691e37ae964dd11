"""Parity at the full workload sizes, in the configuration bench.py times
(all weights and the output head streamed from pinned host memory, 64 MiB
chunks, 3 slots).

The CPU oracle recomputes sampled batch rows at full depth (the rows of a
batch are independent, so a row is a faithful sample of the batch), or every
layer of a short slice of the model; the GPU's other rows are checked by a
property that holds at any size: a row decoded in the full batch matches the
same row decoded alone.
"""
import numpy as np
import pytest

import synth
from oracle import decoder_for
from paper_2504_03664_amd.model import Decoder, HostWeights

pytestmark = pytest.mark.gpu

REL_TOL = 2e-2
# Argmax: every disagreement must be a near tie (check_rows asserts it); of
# the 64 sampled positions at most 5 % may disagree.  Kernels that only
# reorder fp32 sums flip exact near ties (an OPT-13B INT4 run at 1.3e-3
# normwise error had one such flip in 64), so a 99 % bar would demand zero.
ARGMAX_MIN = 0.95
# INT4 KV cache: a code moves by a whole step when a key or value crosses a
# decision boundary, so implementations that differ only in summation order
# differ by far more than with an fp16 cache.  At the OPT-30B slice two
# readings of the oracle itself (expanded INT4 weights kept in fp32 or
# rounded to fp16) differ by 4.2e-2 normwise; the bar is set at 5e-2, with
# argmax disagreements allowed only at near ties of that size.
KV4_TOL = 5e-2


def log(msg):
    print(msg, flush=True)


def normwise(g, o):
    return np.abs(g - o).max(axis=-1) / np.abs(o).max(axis=-1)


def run_gpu(hw, wl, prompt, gen, batch_rows=None):
    with Decoder(hw, max_batch=prompt.shape[0], max_seq=wl.prompt + wl.gen,
                 kv_on_host=wl.kv_on_host, kv_fmt=wl.kv_fmt, chunk_bytes=64 << 20) as dec:
        toks, logits = dec.generate(prompt, gen, want_logits=True)
    logits = np.stack(logits, axis=1)          # [b][gen][V]
    return toks, logits


def check_rows(model, prompt, toks, logits, rows, layers=None, kv_int4=False, tol=REL_TOL):
    """Teacher-forced oracle logits for `rows` at every generated position;
    every argmax disagreement must be a near tie (gap <= tol * max |logit|)."""
    full = np.concatenate([prompt[rows], toks[rows, :-1]], axis=1)
    ref = decoder_for(model, np.float32, kv_int4=kv_int4,
                      fp16_operands=kv_int4).forward(full, layers=layers)
    P = prompt.shape[1]
    worst, agree, total = 0.0, 0, 0
    for i, r in enumerate(rows):
        o = ref[i, P - 1:].astype(np.float64)
        g = logits[r].astype(np.float64)
        e = normwise(g, o)
        worst = max(worst, float(e.max()))
        ga, oa = g.argmax(-1), o.argmax(-1)
        agree += int((ga == oa).sum())
        total += len(ga)
        for s in np.nonzero(ga != oa)[0]:
            gap = o[s, oa[s]] - o[s, ga[s]]
            assert gap <= tol * np.abs(o[s]).max(), f"row {r} step {s}: argmax differs, no tie"
    return worst, agree / total


def _workload(i):
    return synth.WORKLOADS[i]


@pytest.mark.parametrize("widx", [1, 2])
def test_full_depth_sampled_rows(widx):
    """OPT-6.7B (fp16, batch 16) and OPT-13B (int4, batch 32) shapes at full
    depth: GPU batch rows 0 and b-1 against the oracle, all 32 positions."""
    wl = _workload(widx)
    log(f"full size {wl.name}: drawing weights")
    model = synth.SyntheticOPT(wl.shape, seed=synth.DEFAULT_SEED, wfmt=wl.wfmt)
    hw = HostWeights(wl.shape, wl.wfmt, model)
    try:
        prompt = synth.prompt_tokens(wl.batch, wl.prompt, wl.shape.vocab, seed=1, stream=widx)
        log("  GPU generation")
        toks, logits = run_gpu(hw, wl, prompt, wl.gen)
    finally:
        hw.free()
    rows = [0, wl.batch - 1]
    log(f"  oracle on rows {rows} ({wl.shape.n_layers} layers)")
    worst, agree = check_rows(model, prompt, toks, logits, rows)
    log(f"  max normwise error {worst:.3e}, argmax agreement {agree:.4f}")
    assert worst <= REL_TOL and agree >= ARGMAX_MIN


@pytest.mark.parametrize("widx", [6, 7])
def test_llama8b_full_depth_sampled_rows(widx):
    """LLaMA-3.1-8B shape (32 layers, d 4096, 32/8 heads, FFN 14336, vocab
    128256) at full depth, fp16 batch 16 or INT4 batch 32, prompt 512, 32
    tokens: GPU batch rows 0 and b-1 against the oracle at every position."""
    wl = _workload(widx)
    log(f"full size {wl.name}: drawing weights")
    model = synth.SyntheticLlama(wl.shape, seed=synth.DEFAULT_SEED, wfmt=wl.wfmt)
    hw = HostWeights(wl.shape, wl.wfmt, model)
    try:
        prompt = synth.prompt_tokens(wl.batch, wl.prompt, wl.shape.vocab, seed=1, stream=widx)
        log("  GPU generation")
        toks, logits = run_gpu(hw, wl, prompt, wl.gen)
    finally:
        hw.free()
    rows = [0, wl.batch - 1]
    log(f"  oracle on rows {rows} ({wl.shape.n_layers} layers)")
    worst, agree = check_rows(model, prompt, toks, logits, rows)
    log(f"  max normwise error {worst:.3e}, argmax agreement {agree:.4f}")
    # At this shape the oracle's own two readings (fp32 activations, or
    # fp16-rounded operands as the kernels hold them) differ by 6.2e-3
    # normwise, and with 128256 random-weight logits the top two are as
    # close as 3.7e-3 of the largest: argmax flips at near ties are expected
    # (each one is checked to be a near tie above).
    assert worst <= REL_TOL and agree >= ARGMAX_MIN


def test_opt30b_layer_slice():
    """OPT-30B shape (d 7168, 56 heads, FFN 28672, batch 64, prompt 512):
    the first 2 layers plus the head streamed, oracle on rows 0 and 63."""
    wl = _workload(3)
    shape = wl.shape.with_layers(2)
    log("30B slice: drawing weights")
    model = synth.SyntheticOPT(shape, seed=synth.DEFAULT_SEED)
    hw = HostWeights(shape, "fp16", model)
    try:
        prompt = synth.prompt_tokens(wl.batch, wl.prompt, shape.vocab, seed=1, stream=3)
        log("  GPU generation")
        toks, logits = run_gpu(hw, wl, prompt, wl.gen)
    finally:
        hw.free()
    worst, agree = check_rows(model, prompt, toks, logits, [0, wl.batch - 1])
    log(f"  max normwise error {worst:.3e}, argmax agreement {agree:.4f}")
    assert worst <= REL_TOL and agree >= ARGMAX_MIN


@pytest.mark.parametrize("widx", [4, 5])
def test_opt30b_full_offload_layer_slice(widx):
    """OPT-30B shape with INT4 weights and the KV cache in host memory (fp16
    or INT4 rows), batch 128, prompt 512, 32 tokens: the first 2 layers plus
    the head, oracle on rows 0 and 127."""
    wl = _workload(widx)
    shape = wl.shape.with_layers(2)
    log(f"{wl.name}, 2-layer slice: drawing weights")
    model = synth.SyntheticOPT(shape, seed=synth.DEFAULT_SEED, wfmt="int4")
    hw = HostWeights(shape, "int4", model)
    try:
        prompt = synth.prompt_tokens(wl.batch, wl.prompt, shape.vocab, seed=1, stream=widx)
        log("  GPU generation")
        toks, logits = run_gpu(hw, wl, prompt, wl.gen)
    finally:
        hw.free()
    kv4 = wl.kv_fmt == "int4"
    tol = KV4_TOL if kv4 else REL_TOL
    worst, agree = check_rows(model, prompt, toks, logits, [0, wl.batch - 1], kv_int4=kv4, tol=tol)
    log(f"  max normwise error {worst:.3e}, argmax agreement {agree:.4f}")
    assert worst <= tol and agree >= (0.9 if kv4 else ARGMAX_MIN)


def test_opt67b_rows_independent_of_batch():
    """Every row of the full batch-16 run matches the same row run alone
    (different GEMM variants, so equal up to rounding)."""
    wl = _workload(1)
    shape = wl.shape.with_layers(8)
    model = synth.SyntheticOPT(shape, seed=synth.DEFAULT_SEED)
    hw = HostWeights(shape, "fp16", model)
    try:
        prompt = synth.prompt_tokens(wl.batch, wl.prompt, shape.vocab, seed=1, stream=1)
        log("batch-16 run (8 layers)")
        toks, logits = run_gpu(hw, wl, prompt, 8)
        for r in (1, 7, 15):
            log(f"  row {r} alone")
            forced = toks[r:r + 1, :-1]
            with Decoder(hw, max_batch=1, max_seq=wl.prompt + 8, chunk_bytes=64 << 20) as dec:
                t1, l1 = dec.generate(prompt[r:r + 1], 8, want_logits=True, forced=forced)
            l1 = np.stack(l1, axis=1)[0].astype(np.float64)
            e = normwise(logits[r].astype(np.float64), l1)
            assert e.max() <= 5e-3, (r, e.max())
    finally:
        hw.free()
