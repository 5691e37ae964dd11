"""The seeded input generator, pinned to library routines and to its definition."""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("key,ctr", [((123, 456), (0, 0, 0, 0)),
                                     ((0, 0), (7, 0, 0, 0)),
                                     ((2**64 - 1, 2**63 + 5), (2**64 - 2, 3, 9, 11))])
def test_philox_matches_numpy(key, ctr):
    # numpy's Philox is Philox4x64-10 and increments its counter before each
    # block, so its first four outputs are philox(ctr + 1, key).
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                          counter=np.array(ctr, dtype=np.uint64))
    expect = bg.random_raw(4)
    c = list(ctr)
    c[0] = (c[0] + 1) % 2**64
    if c[0] == 0:
        c[1] += 1
    got = synth.philox4x64_10(c, key)
    assert (got == expect).all()


def test_f16_rounding_matches_numpy():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(100000).astype(np.float32) * 0.02,
        rng.standard_normal(10000).astype(np.float32) * 1e-6,      # fp16 subnormals
        (np.arange(1, 2049, dtype=np.float32) + 0.5) * 2.0**-24,   # halfway cases
        np.array([65504.0, 65519.0, 65520.0, -70000.0, 0.0, -0.0], dtype=np.float32),
    ])
    got = np.array([synth.f32_to_f16_bits(v) for v in x], dtype=np.uint16)
    assert (got == x.astype(np.float16).view(np.uint16)).all()


def test_normal_stream_statistics():
    z = synth.normal_f16(7, 99, 1 << 22, std=1.0).astype(np.float64)
    assert abs(z.mean()) < 3e-3
    assert abs(z.std() - 1.0) < 3e-3
    assert abs(np.mean(np.abs(z) < 1.0) - 0.682689) < 2e-3
    assert abs(np.mean(np.abs(z) < 2.0) - 0.954500) < 1e-3
    w = synth.normal_f16(7, 100, 1 << 20).astype(np.float64)
    assert abs(w.std() - 0.02) < 1e-4


def test_stream_is_counter_based():
    full = synth.normal_f16(3, 5, 5000)
    part = synth.normal_f16(3, 5, 777, first=1234)
    assert (part.view(np.uint16) == full[1234:2011].view(np.uint16)).all()
    other = synth.normal_f16(3, 6, 5000)
    assert (other.view(np.uint16) != full.view(np.uint16)).mean() > 0.99
    again = synth.normal_f16(3, 5, 5000)
    assert (again.view(np.uint16) == full.view(np.uint16)).all()


def test_int4_encoding_definition():
    w = synth.normal_f16(1, 2, 8 * 256).reshape(8, 256)
    q, sm = synth.quant_int4_g64(w)
    assert q.shape == (8, 128) and sm.shape == (8, 4, 2)
    wf = w.astype(np.float32).reshape(8, 4, 64)
    mn, mx = wf.min(-1), wf.max(-1)
    assert (sm[..., 0] == ((mx - mn) / np.float32(15)).astype(np.float16)).all()
    assert (sm[..., 1] == mn.astype(np.float16)).all()
    codes = np.empty((8, 256), dtype=np.int64)
    codes[:, 0::2] = q & 15
    codes[:, 1::2] = q >> 4
    s = sm[..., 0].astype(np.float32)[..., None]
    m = sm[..., 1].astype(np.float32)[..., None]
    expect = np.clip(np.rint((wf - m) / s), 0, 15)
    assert (codes.reshape(8, 4, 64) == expect).all()


def test_fused_int4_equals_encode_of_draw():
    N, K = 33, 192
    q, sm = synth.normal_int4_g64(11, 12, N, K)
    w = synth.normal_f16(11, 12, N * K).reshape(N, K)
    q2, sm2 = synth.quant_int4_g64(w)
    assert (q == q2).all() and (sm.view(np.uint16) == sm2.view(np.uint16)).all()


def test_prompt_tokens():
    t = synth.prompt_tokens(4, 32, 50272, seed=1)
    assert t.dtype == np.int32 and t.shape == (4, 32)
    assert t.min() >= 0 and t.max() < 50272
    assert (t == synth.prompt_tokens(4, 32, 50272, seed=1)).all()
    assert (t != synth.prompt_tokens(4, 32, 50272, seed=2)).any()


def test_synthetic_model_layout():
    m = synth.SyntheticOPT(synth.OPTShape(2, 64, 4, 256, vocab=100, max_pos=16))
    L = m.layer(1)
    assert L["wqkv"].shape == (192, 64) and L["w2"].shape == (64, 256)
    assert (L["ln1_g"] == 1).all() and (L["ln2_b"] == 0).all()
    assert L["bqkv"].std() > 0.01
    assert m.tok_emb().shape == (100, 64) and m.pos_emb().shape == (18, 64)
    m4 = synth.SyntheticOPT(m.shape, wfmt="int4")
    q, sm = m4.layer(1)["w1"]
    q2, sm2 = synth.quant_int4_g64(L["w1"])
    assert (q == q2).all() and (sm.view(np.uint16) == sm2.view(np.uint16)).all()


def test_teacher_tokens_are_seeded_and_independent():
    wl = synth.WORKLOADS[1]
    p, f = synth.teacher_tokens(wl, stream=1)
    assert p.shape == (wl.batch, wl.prompt) and f.shape == (wl.batch, wl.gen - 1)
    assert p.min() >= 0 and f.max() < wl.shape.vocab
    p2, f2 = synth.teacher_tokens(wl, stream=1)
    assert (p == p2).all() and (f == f2).all()
    assert (f != p[:, :wl.gen - 1]).any()
    assert (synth.teacher_tokens(wl, stream=2)[1] != f).any()


@pytest.mark.parametrize("wfmt", ["fp16", "int4"])
def test_zero_kv_provider(wfmt):
    """ZeroKV zeroes exactly the key and value rows of wqkv (an INT4 zero
    row: codes 0, scale 0, min 0) in every access path; the query rows and
    every other tensor are the base provider's."""
    base = synth.SyntheticOPT(synth.OPTShape(2, 128, 2, 256, vocab=100, max_pos=16), wfmt=wfmt)
    z = synth.ZeroKV(base)
    d = 128
    Lb, Lz = base.layer(1), z.layer(1)
    for nm in ("wo", "w1", "w2", "bqkv", "ln1_g"):
        a, b = Lb[nm], Lz[nm]
        if isinstance(a, tuple):
            assert all(np.array_equal(x.view(np.uint8), y.view(np.uint8)) for x, y in zip(a, b))
        else:
            assert np.array_equal(a.view(np.uint16), b.view(np.uint16))
    if wfmt == "fp16":
        w = Lz["wqkv"]
        assert np.array_equal(w[:d].view(np.uint16), Lb["wqkv"][:d].view(np.uint16))
        assert (w[d:] == 0).all()
        out = z.fill(1, "wqkv", np.empty((3 * d, d), np.float16))
        assert np.array_equal(out.view(np.uint16), w.view(np.uint16))
    else:
        q, sm = Lz["wqkv"]
        assert np.array_equal(q[:d], Lb["wqkv"][0][:d]) and (q[d:] == 0).all()
        assert (sm[d:].view(np.uint16) == 0).all()
        q2 = np.empty_like(q)
        sm2 = np.empty_like(sm)
        z.fill_int4(1, "wqkv", q2, sm2)
        assert np.array_equal(q2, q) and np.array_equal(sm2.view(np.uint16), sm.view(np.uint16))
