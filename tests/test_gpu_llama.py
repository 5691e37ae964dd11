"""The LLaMA-3.1-style decoder end to end on the GPU against the oracle
(teacher forced), and the pipelined runs against the same kernels with
every weight resident in HBM (bit for bit)."""
import numpy as np
import pytest

import synth
from oracle import LlamaDecoder
from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.model import Decoder, HostWeights, c_policy, c_shape

pytestmark = pytest.mark.gpu

REL_TOL = 2e-2          # normwise per logits row: max|g - o| / max|o|
KV4_TOL = 5e-2          # INT4 cache with real key/value projections: code flips between
                        # implementations that differ only in summation order
ARGMAX_MIN = 0.99

# head_dim 64, 4 query heads per key/value head (dkv 128); prompts with a
# ragged prefill tile
SMALL64 = synth.LlamaShape(3, 512, 8, 2, 1024, vocab=1000, max_pos=256)
# head_dim 128, 4 query heads per key/value head (dkv 256: INT4 cache rows)
SMALL128 = synth.LlamaShape(3, 1024, 8, 2, 1536, vocab=1500, max_pos=256)
# 8 query heads per key/value head, no frequency scaling
SMALL_G8 = synth.LlamaShape(2, 1024, 16, 2, 1024, vocab=700, max_pos=128, rope_theta=10000.0,
                            rope_factor=0.0)


def log(msg):
    print(msg, flush=True)


def normwise(g, o):
    return np.abs(g - o).max(axis=-1) / np.abs(o).max(axis=-1)


def _model(shape, seed, wfmt="fp16"):
    # random RMSNorm gains, so that a norm reading the wrong gain shows
    return synth.SyntheticLlama(shape, seed=seed, wfmt=wfmt, gain_std=0.2)


def forced_tokens(prompt, gen, vocab):
    """The ids fed at the gen - 1 decode steps of a teacher-forced run
    (seeded, a function of the prompt's shape), so that the oracle's inputs
    never come from the GPU."""
    b, P = prompt.shape
    return synth.prompt_tokens(b, gen - 1, vocab, seed=3, stream=P * 1000 + b)


def _run(hw, prompt, gen, **pol):
    """A teacher-forced run: tokens [b][gen], logits [gen][b][V]."""
    forced = forced_tokens(prompt, gen, hw.shape.vocab)
    with Decoder(hw, max_batch=prompt.shape[0], max_seq=prompt.shape[1] + gen, **pol) as dec:
        toks, logits = dec.generate(prompt, gen, want_logits=True, forced=forced)
    return toks, np.stack(logits)


def teacher_forced_check(model, prompt, toks, logits, kv_int4=False, tol=REL_TOL):
    """Oracle logits at every generated position of a teacher-forced run.
    The normwise error is taken against the plain fp32 oracle; the greedy
    tokens against the reading that keeps the paper's fp16 activations
    (Section 4.1), the precision in which the kernels decide them; every
    disagreement must be a near tie.  With an INT4 cache both use that
    reading (its codes are decided on the same fp16 keys and values as the
    kernels').  Returns (worst normwise error, agreement, near ties, the
    agreement of the oracle's fp32 and fp16-activation readings)."""
    gen = toks.shape[1]
    full = np.concatenate([prompt, forced_tokens(prompt, gen, model.shape.vocab)], axis=1)
    ref32 = LlamaDecoder(model, np.float32, kv_int4=kv_int4).forward(full, last=gen)
    ref16 = LlamaDecoder(model, np.float32, kv_int4=kv_int4,
                         fp16_operands=True).forward(full, last=gen)
    ref = ref16 if kv_int4 else ref32
    worst, agree, total, ties = 0.0, 0, 0, 0
    for s in range(gen):
        o = ref[:, s].astype(np.float64)
        o16 = ref16[:, s].astype(np.float64)
        g = logits[s].astype(np.float64)
        worst = max(worst, float(normwise(g, o).max()))
        ga, oa = g.argmax(-1), o16.argmax(-1)
        assert (ga == toks[:, s]).all()
        agree += int((ga == oa).sum())
        total += len(ga)
        for r in np.nonzero(ga != oa)[0]:
            assert o16[r, oa[r]] - o16[r, ga[r]] <= tol * np.abs(o16[r]).max(), \
                "argmax, no near tie"
            ties += 1
    own = float((ref32.argmax(-1) == ref16.argmax(-1)).mean())
    return worst, agree / total, ties, own


@pytest.mark.parametrize("shape,wfmt", [(SMALL64, "fp16"), (SMALL128, "fp16"),
                                        (SMALL128, "int4"), (SMALL_G8, "fp16")])
def test_llama_streamed_parity_and_resident_identity(shape, wfmt):
    """Every layer and the untied head streamed per matrix: against the
    oracle, and bit-identical to the run with everything resident and to
    other pipelines (one slot, two slots with small chunks, host KV)."""
    log(f"llama d={shape.d_model} h={shape.n_heads}/{shape.n_kv_heads} {wfmt}")
    model = _model(shape, seed=21, wfmt=wfmt)
    hw = HostWeights(shape, wfmt, model)
    try:
        prompt = synth.prompt_tokens(3, 37, shape.vocab, seed=4)
        t0, l0 = _run(hw, prompt, 8, chunk_bytes=1 << 20)
        err, agree, ties, _ = teacher_forced_check(model, prompt, t0, l0)
        log(f"  err {err:.2e} agree {agree:.3f} ({ties} near ties)")
        assert err <= REL_TOL and agree >= ARGMAX_MIN
        for v in (dict(weights_on_host=False, embed_on_host=False),
                  dict(embed_on_host=False),
                  dict(n_weight_slots=1),
                  dict(n_weight_slots=2, chunk_bytes=4096 * 37, n_h2d_streams=1),
                  dict(debug_flags=B.PIPO_DBG_SEGMENT_COPIES),
                  dict(debug_flags=B.PIPO_DBG_UNFUSED),   # SwiGLU as its own kernel
                  dict(kv_on_host=True, debug_flags=B.PIPO_DBG_POISON_SLOTS),
                  dict(kv_on_host=True, n_weight_slots=1, chunk_bytes=1 << 18)):
            log(f"  variant {v}")
            tv, lv = _run(hw, prompt, 8, **v)
            assert np.array_equal(tv, t0)
            assert np.array_equal(lv.view(np.uint32), l0.view(np.uint32))
    finally:
        hw.free()


def test_llama_int4_disk_tier(tmp_path):
    """INT4 LLaMA layers streamed from the disk tier, bit-identical to the
    resident run."""
    model = _model(SMALL128, seed=25, wfmt="int4")
    hw = HostWeights(SMALL128, "int4", model)
    try:
        prompt = synth.prompt_tokens(2, 40, SMALL128.vocab, seed=7)
        t0, l0 = _run(hw, prompt, 5, weights_on_host=False, embed_on_host=False)
        t1, l1 = _run(hw, prompt, 5, weights_on_disk=True, disk_dir=str(tmp_path),
                      chunk_bytes=1 << 20)
        assert np.array_equal(t1, t0)
        assert np.array_equal(l1.view(np.uint32), l0.view(np.uint32))
    finally:
        hw.free()


@pytest.mark.parametrize("wfmt", ["fp16", "int4"])
def test_llama_int4_kv_cache(wfmt):
    """INT4 cache rows (keys quantized after their rotation) against the
    oracle with the same cache format, and bit-identical with the cache in
    host memory (pinned, and pageable through the staging rings)."""
    log(f"llama int4 kv, {wfmt} weights")
    model = _model(SMALL128, seed=22, wfmt=wfmt)
    hw = HostWeights(SMALL128, wfmt, model)
    try:
        prompt = synth.prompt_tokens(4, 70, SMALL128.vocab, seed=5)
        t0, l0 = _run(hw, prompt, 8, kv_fmt="int4")
        err, agree, ties, own = teacher_forced_check(model, prompt, t0, l0, kv_int4=True,
                                                     tol=KV4_TOL)
        log(f"  err {err:.2e} agree {agree:.3f} ({ties} near ties); the oracle's fp32 and "
            f"fp16-activation readings agree on {own:.3f}")
        # With an INT4 cache a key or value within rounding of a code
        # boundary takes a different code on each side (the fp32 summation
        # order decides which), so the GPU is held to the 99 % bar or, where
        # the oracle's own two readings agree less, to theirs; every
        # disagreement was checked to be a near tie at KV4_TOL.
        assert err <= KV4_TOL and agree >= min(ARGMAX_MIN, own)
        for v in (dict(weights_on_host=False, embed_on_host=False),
                  dict(kv_on_host=True),
                  dict(kv_on_host=True, debug_flags=B.PIPO_DBG_KV_PAGEABLE, chunk_bytes=1 << 16)):
            log(f"  variant {v}")
            tv, lv = _run(hw, prompt, 8, kv_fmt="int4", **v)
            assert np.array_equal(tv, t0)
            assert np.array_equal(lv.view(np.uint32), l0.view(np.uint32))
    finally:
        hw.free()


def test_llama_longer_generation_crosses_prefill_tiles():
    """Prompt 130 (three 64-row prefill tiles, ragged) and 40 decode steps."""
    log("llama p130 g40")
    model = _model(SMALL64, seed=23)
    hw = HostWeights(SMALL64, "fp16", model)
    try:
        prompt = synth.prompt_tokens(2, 130, SMALL64.vocab, seed=6)
        t0, l0 = _run(hw, prompt, 40)
        err, agree, ties, _ = teacher_forced_check(model, prompt, t0, l0)
        log(f"  err {err:.2e} agree {agree:.3f}")
        assert err <= REL_TOL and agree >= ARGMAX_MIN
    finally:
        hw.free()


def test_llama_planned_memory_is_allocated_memory():
    log("llama memory plan vs allocation")
    model = _model(SMALL128, seed=24)
    hw = HostWeights(SMALL128, "fp16", model)
    try:
        shape = c_shape(SMALL128)
        for pol in (dict(), dict(weights_on_host=False, embed_on_host=False),
                    dict(embed_on_host=False, kv_fmt="int4", n_weight_slots=2),
                    dict(kv_on_host=True, n_weight_slots=1)):
            pol = dict(dict(max_batch=3, max_seq=50), **pol)
            want = B.pipo_plan_policy(shape, c_policy(**pol))["hbm_bytes"]
            with Decoder(hw, **pol) as dec:
                assert dec.stats()["hbm_bytes"] == want, pol
    finally:
        hw.free()
