"""Host-side parts of the LLaMA-family path, without a GPU: the rotary table
the library uploads, shape validation, and the memory plan against the
paper's size formulas (Section 3.5)."""
import numpy as np
import pytest

import synth
from oracle import llama_kv_bytes, llama_param_count, rope_frequencies
from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.model import c_policy, c_shape


def _oracle_table(shape, n_pos):
    w = rope_frequencies(shape.head_dim, shape.rope_theta, shape.rope_factor,
                         shape.rope_low_freq_factor, shape.rope_high_freq_factor,
                         shape.rope_orig_max_pos)
    ang = np.arange(n_pos, dtype=np.float64)[:, None] * w[None, :]
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1)


@pytest.mark.parametrize("shape", [
    synth.LLAMA31_8B,                                                  # 3.1 scaling, dh 128
    synth.LlamaShape(2, 512, 8, 2, 1024, vocab=100, rope_theta=10000.0, rope_factor=0.0),
    synth.LlamaShape(2, 256, 4, 4, 512, vocab=100, rope_factor=4.0, rope_low_freq_factor=2.0,
                     rope_high_freq_factor=8.0, rope_orig_max_pos=1024),
])
def test_rope_table_matches_oracle_frequencies(shape):
    """The library's (cos, sin) table is the oracle's angles, rounded once to
    fp32 (both sides compute in double)."""
    n_pos = 4096
    got = B.pipo_rope_table(c_shape(shape), n_pos).astype(np.float64)
    want = _oracle_table(shape, n_pos)
    ulp = np.spacing(np.abs(want).astype(np.float32)).astype(np.float64)
    assert (np.abs(got - want) <= ulp).all()


def test_rope_table_scaling_changes_only_low_frequencies():
    """With the 3.1 scaling, the high-frequency components (wavelength below
    orig / high_freq_factor) keep their unscaled angles."""
    sh = synth.LLAMA31_8B
    plain = synth.LlamaShape(1, sh.d_model, sh.n_heads, sh.n_kv_heads, sh.d_ffn, vocab=10,
                             rope_factor=0.0)
    a = B.pipo_rope_table(c_shape(sh), 512)
    b = B.pipo_rope_table(c_shape(plain), 512)
    w = rope_frequencies(sh.head_dim, sh.rope_theta)
    short = 2 * np.pi / w < sh.rope_orig_max_pos / sh.rope_high_freq_factor
    assert short.any() and not short.all()
    assert np.array_equal(a[:, short], b[:, short])
    assert not np.array_equal(a[1:, ~short], b[1:, ~short])


def _status(fn):
    with pytest.raises(B.PipoError) as e:
        fn()
    return B.STATUS_NAMES[e.value.status]


def test_shape_validation():
    pol = c_policy(max_batch=1, max_seq=8)
    plan = lambda sh: B.pipo_plan_policy(sh, pol)  # noqa: E731
    ok = c_shape(synth.LlamaShape(2, 512, 8, 2, 1024, vocab=100))
    plan(ok)
    bad = c_shape(synth.LlamaShape(2, 512, 8, 3, 1024, vocab=100))   # 8 % 3 != 0
    assert _status(lambda: plan(bad)) == "PIPO_ERR_ARG"
    g3 = c_shape(synth.LlamaShape(2, 768, 12, 4, 1024, vocab=100))   # 3 query heads per kv head
    assert _status(lambda: plan(g3)) == "PIPO_ERR_UNSUPPORTED"
    no_theta = c_shape(synth.LlamaShape(2, 512, 8, 2, 1024, vocab=100))
    no_theta.rope_theta = 0.0
    assert _status(lambda: plan(no_theta)) == "PIPO_ERR_ARG"
    bad_scale = c_shape(synth.LlamaShape(2, 512, 8, 2, 1024, vocab=100))
    bad_scale.rope_high_freq_factor = bad_scale.rope_low_freq_factor
    assert _status(lambda: plan(bad_scale)) == "PIPO_ERR_ARG"
    opt_gqa = c_shape(synth.OPT_125M)
    opt_gqa.n_kv_heads = 6   # 2 query heads per kv head
    assert _status(lambda: plan(opt_gqa)) == "PIPO_ERR_ARG"
    fam = c_shape(synth.OPT_125M)
    fam.family = 7
    assert _status(lambda: plan(fam)) == "PIPO_ERR_ARG"
    # an INT4 cache needs cached rows of a multiple of 256 elements
    narrow = c_shape(synth.LlamaShape(2, 512, 8, 1, 1024, vocab=100))   # dkv = 64
    assert _status(lambda: B.pipo_plan_policy(narrow, c_policy(max_batch=1, max_seq=8,
                                                               kv_fmt="int4"))) \
        == "PIPO_ERR_UNSUPPORTED"


@pytest.mark.parametrize("shape", [synth.LLAMA31_8B, synth.LLAMA31_70B])
def test_plan_matches_the_papers_size_formulas(shape):
    """Section 3.5: W = 2 W_embed + l (W_mha + W_mlp) elements and C = 2 p b s
    l d h_kv / h bytes; the library's plan holds exactly these bytes (fp16)."""
    cs = c_shape(shape)
    b, s = 16, 544
    plan = B.pipo_plan_policy(cs, c_policy(max_batch=b, max_seq=s))
    W = llama_param_count(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads,
                          shape.d_ffn, shape.vocab)
    assert plan["weight_bytes"] == 2 * W
    assert plan["kv_bytes"] == llama_kv_bytes(shape.n_layers, shape.d_model, shape.n_heads,
                                              shape.n_kv_heads, b, s)
    # INT4 cache rows: 9 dkv / 16 bytes instead of 2 dkv
    plan4 = B.pipo_plan_policy(cs, c_policy(max_batch=b, max_seq=s, kv_fmt="int4"))
    assert plan4["kv_bytes"] * 32 == plan["kv_bytes"] * 9


def test_streamed_bytes_per_step():
    """A decode step with everything streamed moves every layer and the
    untied head once (plus the token rows gathered on the host); each
    layer's two norm gains (2 d fp16 values) travel in a copy padded to 32
    KiB, the shortest copy the runtime gives to a DMA engine."""
    sh = synth.LLAMA31_8B
    b, s = 16, 544
    plan = B.pipo_plan_policy(c_shape(sh), c_policy(max_batch=b, max_seq=s))
    W = llama_param_count(sh.n_layers, sh.d_model, sh.n_heads, sh.n_kv_heads, sh.d_ffn, sh.vocab)
    tok_table, final_norm = sh.vocab * sh.d_model, sh.d_model
    pad = sh.n_layers * max(0, 32768 - 2 * 2 * sh.d_model)
    assert plan["h2d_bytes_per_step"] == 2 * (W - tok_table - final_norm) + b * sh.d_model * 2 \
        + b * 4 + pad
