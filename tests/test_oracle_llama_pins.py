"""Pins for the LLaMA-3.1-style oracle: the paper's size formulas, hand
values, closed forms and invariants of rotary positions, grouped-query
attention reduced to plain multi-head attention, a scalar brute-force
decoder, and incremental decoding against full recomputation."""
import json
import math
import os
import types

import numpy as np
import pytest

import synth
from oracle import (LlamaDecoder, apply_rope, causal_attention, gqa_attention, llama_kv_bytes,
                    llama_param_count, rms_norm, rope_frequencies)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_weight_size_against_the_paper():
    """Section 3.5's W = 2 W_embed + l (W_mha + W_mlp) for LLaMA3.1-8B in fp16
    is 'more than 16 GB' (Section 4.2); 70B comes to ~141 GB."""
    with open(os.path.join(GOLDEN, "paper_weight_sizes.json")) as f:
        fact = json.load(f)["llama3_1_8b_fp16_weight_gb_more_than"]
    s = synth.LLAMA31_8B
    n8 = llama_param_count(s.n_layers, s.d_model, s.n_heads, s.n_kv_heads, s.d_ffn, s.vocab)
    assert 2 * n8 / 1e9 > fact["value"]
    # written out: embedding and head 2 x 525,336,576, 32 layers of
    # 218,112,000 (q, o, the 8-head k and v, norm; gate, up, down, norm), final norm
    assert n8 == 2 * 128256 * 4096 + 32 * (4096 * (8192 + 2048 + 1) + 4096 * (3 * 14336 + 1)) + 4096
    assert n8 == 8_030_261_248
    s = synth.LLAMA31_70B
    n70 = llama_param_count(s.n_layers, s.d_model, s.n_heads, s.n_kv_heads, s.d_ffn, s.vocab)
    assert abs(2 * n70 / 1e9 - 141.1) < 0.1


def test_kv_size_formula():
    """C = 2 p b s l d h_kv / h: K and V rows of h_kv heads."""
    assert llama_kv_bytes(32, 4096, 32, 8, 16, 544) == 2 * 2 * 16 * 544 * 32 * 1024


def test_rms_norm_hand_values():
    x = np.array([3.0, -4.0, 0.0, 0.0])
    # mean of squares 25/4, rms 2.5
    got = rms_norm(x, np.array([1.0, 1.0, 2.0, 0.5]), 0.0)
    assert np.allclose(got, [1.2, -1.6, 0.0, 0.0])
    got = rms_norm(np.array([1.0, 1.0]), np.array([1.0, 1.0]), 3.0)   # 1 / sqrt(1 + 3)
    assert np.allclose(got, [0.5, 0.5])


def test_rope_frequencies_closed_forms():
    w = rope_frequencies(8, 10000.0)
    assert np.allclose(w, [1.0, 10000 ** -0.25, 10000 ** -0.5, 10000 ** -0.75])
    base = rope_frequencies(128, 500000.0)
    scaled = rope_frequencies(128, 500000.0, 8.0, 1.0, 4.0, 8192)
    wl = 2 * np.pi / base
    short = wl < 8192 / 4
    long = wl > 8192 / 1
    assert short.any() and long.any() and (~short & ~long).any()
    assert np.array_equal(scaled[short], base[short])                  # high frequencies kept
    assert np.allclose(scaled[long], base[long] / 8)                   # low ones divided by 8
    mid = ~short & ~long
    assert ((scaled[mid] < base[mid]) & (scaled[mid] > base[mid] / 8)).all()
    # the blend meets both branches at its ends (s = 0 at wavelength 8192, 1 at 2048)
    for lam, want in ((8192.0, 1 / 8), (2048.0, 1.0)):
        w0 = 2 * np.pi / lam
        s = (8192 / lam - 1) / 3
        assert np.isclose((1 - s) * w0 / 8 + s * w0, w0 * want)


def test_rope_rotation_properties():
    rng = np.random.default_rng(0)
    freqs = rope_frequencies(8, 10000.0)
    x = rng.standard_normal((5, 16))                                  # 2 heads of 8
    pos = np.array([0, 1, 7, 100, 4096])
    y = apply_rope(x, pos, freqs)
    assert np.allclose(y[0], x[0])                                    # position 0: identity
    for hd in range(2):                                               # pair norms kept
        a = x[:, hd * 8:hd * 8 + 4] ** 2 + x[:, hd * 8 + 4:hd * 8 + 8] ** 2
        b = y[:, hd * 8:hd * 8 + 4] ** 2 + y[:, hd * 8 + 4:hd * 8 + 8] ** 2
        assert np.allclose(a, b)
    # a unit vector in the first slot of the first pair turns to (cos, sin)
    e = np.zeros((1, 8))
    e[0, 0] = 1
    r = apply_rope(e, np.array([3]), freqs)[0]
    assert np.allclose([r[0], r[4]], [math.cos(3.0), math.sin(3.0)]) and np.allclose(r[[1, 2, 3, 5, 6, 7]], 0)
    # scores depend only on the distance between positions
    q, k = rng.standard_normal((1, 8)), rng.standard_normal((1, 8))
    dot = lambda m, n: (apply_rope(q, np.array([m]), freqs) @ apply_rope(k, np.array([n]), freqs).T)[0, 0]  # noqa: E731
    assert np.isclose(dot(10, 3), dot(17, 10)) and np.isclose(dot(5, 5), (q @ k.T)[0, 0])


def test_gqa_reduces_to_multi_head_attention():
    rng = np.random.default_rng(1)
    T, S, h, hkv, dh = 3, 6, 4, 2, 8
    q = rng.standard_normal((T, h * dh))
    k = rng.standard_normal((S, hkv * dh))
    v = rng.standard_normal((S, hkv * dh))
    # repeat every key/value head for its group of query heads
    rep = lambda a: np.concatenate([a[:, (j // 2) * dh:(j // 2 + 1) * dh] for j in range(h)], axis=1)  # noqa: E731
    assert np.allclose(gqa_attention(q, k, v, h, hkv), causal_attention(q, rep(k), rep(v), h))
    k2 = rng.standard_normal((S, h * dh))
    v2 = rng.standard_normal((S, h * dh))
    assert np.allclose(gqa_attention(q, k2, v2, h, h), causal_attention(q, k2, v2, h))


def small_model(L=2, d=16, h=4, hkv=2, F=24, V=11, seed=0, scale=0.4):
    shape = types.SimpleNamespace(n_layers=L, d_model=d, n_heads=h, n_kv_heads=hkv, d_ffn=F,
                                  vocab=V, ln_eps=1e-5, head_dim=d // h, rope_theta=10000.0,
                                  rope_factor=0.0, rope_low_freq_factor=1.0,
                                  rope_high_freq_factor=4.0, rope_orig_max_pos=8192,
                                  family="llama")
    rng = np.random.default_rng(seed)
    dh = d // h
    layers = [dict(ln1_g=1 + 0.1 * rng.standard_normal(d),
                   wqkv=rng.standard_normal(((h + 2 * hkv) * dh, d)) * scale,
                   wo=rng.standard_normal((d, d)) * scale,
                   ln2_g=1 + 0.1 * rng.standard_normal(d),
                   w1=rng.standard_normal((2 * F, d)) * scale,
                   w2=rng.standard_normal((d, F)) * scale) for _ in range(L)]
    tok = rng.standard_normal((V, d))
    head = rng.standard_normal((V, d)) * scale
    lnf = 1 + 0.1 * rng.standard_normal(d)
    return types.SimpleNamespace(shape=shape, wfmt="fp16", layer=lambda j: layers[j],
                                 tok_emb=lambda: tok, lm_head=lambda: head, lnf=lambda: (lnf, None),
                                 layers=layers, tok=tok, head=head, lnf_g=lnf)


def brute_llama(w, tokens):
    """Scalar-loop forward of one sequence (float64, math only)."""
    s = w.shape
    d, h, hkv, F = s.d_model, s.n_heads, s.n_kv_heads, s.d_ffn
    dh, half, grp = d // h, d // h // 2, h // hkv
    T = len(tokens)

    def rms(vec, g):
        r = math.sqrt(sum(a * a for a in vec) / d + s.ln_eps)
        return [vec[c] / r * g[c] for c in range(d)]

    def lin(W, vec):
        return [sum(W[r][c] * vec[c] for c in range(len(vec))) for r in range(len(W))]

    def rot(vec, p, heads):
        out = list(vec)
        for hh in range(heads):
            for i in range(half):
                ang = p * s.rope_theta ** (-2 * i / dh)
                a, b = vec[hh * dh + i], vec[hh * dh + i + half]
                out[hh * dh + i] = a * math.cos(ang) - b * math.sin(ang)
                out[hh * dh + i + half] = b * math.cos(ang) + a * math.sin(ang)
        return out

    xs = [list(w.tok[t]) for t in tokens]
    for L in w.layers:
        qs, ks, vs = [], [], []
        for p, x in enumerate(xs):
            qkv = lin(L["wqkv"], rms(x, L["ln1_g"]))
            qs.append(rot([a / math.sqrt(dh) for a in qkv[:h * dh]], p, h))
            ks.append(rot(qkv[h * dh:(h + hkv) * dh], p, hkv))
            vs.append(qkv[(h + hkv) * dh:])
        new = []
        for i in range(T):
            o = [0.0] * d
            for hh in range(h):
                kh = hh // grp
                sc = [sum(qs[i][hh * dh + c] * ks[j][kh * dh + c] for c in range(dh)) for j in range(i + 1)]
                m = max(sc)
                e = [math.exp(a - m) for a in sc]
                for c in range(dh):
                    o[hh * dh + c] = sum(e[j] * vs[j][kh * dh + c] for j in range(i + 1)) / sum(e)
            x = [xs[i][c] + v for c, v in enumerate(lin(L["wo"], o))]
            gu = lin(L["w1"], rms(x, L["ln2_g"]))
            hid = [gu[n] / (1 + math.exp(-gu[n])) * gu[F + n] for n in range(F)]
            new.append([x[c] + v for c, v in enumerate(lin(L["w2"], hid))])
        xs = new
    return np.array([lin(w.head, rms(x, w.lnf_g)) for x in xs])


def test_decoder_vs_scalar_brute_force():
    w = small_model()
    toks = np.array([[3, 1, 4, 1, 5], [9, 2, 6, 5, 3]])
    got = LlamaDecoder(w, np.float64).forward(toks)
    for b in range(2):
        assert np.allclose(got[b], brute_llama(w, list(toks[b])), rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("kv_int4,fp16_ops", [(False, False), (True, False), (True, True)])
def test_incremental_decode_equals_full_recompute(kv_int4, fp16_ops):
    w = small_model(d=256, h=4, hkv=2, F=64, V=13, seed=2, scale=0.08)
    toks = np.array([[1, 2, 3, 4, 5, 6, 7], [7, 6, 5, 4, 3, 2, 1]])
    dec = LlamaDecoder(w, np.float64, kv_int4=kv_int4, fp16_operands=fp16_ops)
    full = dec.forward(toks)
    P = 3
    logits, cache = dec.prefill(toks[:, :P])
    assert np.allclose(logits, full[:, P - 1], rtol=1e-12, atol=1e-12)
    for t in range(P, toks.shape[1]):
        assert np.allclose(dec.decode(cache, toks[:, t]), full[:, t], rtol=1e-12, atol=1e-12)


def test_causality():
    w = small_model(seed=4)
    toks = np.array([[1, 2, 3, 4, 5, 6]])
    dec = LlamaDecoder(w, np.float64)
    base = dec.forward(toks)[0]
    pert = toks.copy()
    pert[0, 3] = 9
    out = dec.forward(pert)[0]
    assert np.array_equal(out[:3], base[:3]) and not np.allclose(out[3:], base[3:])
