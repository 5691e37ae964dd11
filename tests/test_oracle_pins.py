"""Pins for the CPU oracle: closed forms, hand-derived values, brute force on
tiny inputs, and invariants of the decoder definition.  Each test is chosen
so that a plausible slip in the oracle (a dropped term, a wrong sign, index or
offset, a transposed operand) makes it fail."""
import json
import math
import os
import types

import numpy as np
import pytest

import synth
from oracle import (OracleDecoder, causal_attention, decoder_for, dequant_int4_g64, layer_norm,
                    param_count, quant_kv_int4_g64, streamed_bytes_per_step)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


class HandWeights:
    """Weight provider built from explicit arrays (float64)."""

    def __init__(self, d, h, F, V, L, n_pos_rows, pos_offset=2, eps=0.0):
        self.shape = types.SimpleNamespace(n_layers=L, d_model=d, n_heads=h, d_ffn=F, vocab=V,
                                           pos_offset=pos_offset, ln_eps=eps)
        self.wfmt = "fp16"
        z = np.zeros
        self.tok = z((V, d))
        self.pos = z((n_pos_rows, d))
        self.lnf_g, self.lnf_b = np.ones(d), z(d)
        self.layers = [dict(ln1_g=np.ones(d), ln1_b=z(d), wqkv=z((3 * d, d)), bqkv=z(3 * d),
                            wo=z((d, d)), bo=z(d), ln2_g=np.ones(d), ln2_b=z(d),
                            w1=z((F, d)), b1=z(F), w2=z((d, F)), b2=z(d)) for _ in range(L)]

    def tok_emb(self):
        return self.tok

    def pos_emb(self):
        return self.pos

    def lnf(self):
        return self.lnf_g, self.lnf_b

    def layer(self, j):
        return self.layers[j]


def random_hand(d=8, h=2, F=16, V=11, L=2, n_pos=12, seed=0, scale=0.5):
    rng = np.random.default_rng(seed)
    w = HandWeights(d, h, F, V, L, n_pos, eps=1e-5)
    w.tok = rng.standard_normal((V, d)) * scale
    w.pos = rng.standard_normal((n_pos, d)) * scale
    w.lnf_g = 1 + 0.1 * rng.standard_normal(d)
    w.lnf_b = 0.1 * rng.standard_normal(d)
    for lw in w.layers:
        for k in list(lw):
            lw[k] = lw[k] + rng.standard_normal(lw[k].shape) * scale
    return w


# ---------------------------------------------------------------------------
# LayerNorm
def test_layer_norm_hand_values():
    # x = [1, 2, 3, 4]: mean 2.5, population variance 1.25
    x = np.array([1.0, 2.0, 3.0, 4.0])
    y = layer_norm(x, np.ones(4), np.zeros(4), 0.0)
    inv = 1 / math.sqrt(1.25)
    assert np.allclose(y, [-1.5 * inv, -0.5 * inv, 0.5 * inv, 1.5 * inv], rtol=0, atol=1e-15)
    # gamma, beta and eps enter as gamma * (x - mu) / sqrt(var + eps) + beta
    y = layer_norm(x, np.array([2.0, 1, 1, 1]), np.array([0, 0, 0, 0.5]), 0.75)
    assert np.allclose(y, [-3.0 / math.sqrt(2), -0.5 / math.sqrt(2), 0.5 / math.sqrt(2),
                           1.5 / math.sqrt(2) + 0.5], atol=1e-15)
    r = layer_norm(np.random.default_rng(1).standard_normal((5, 64)) * 3 + 7,
                   np.ones(64), np.zeros(64), 0.0)
    assert np.allclose(r.mean(-1), 0, atol=1e-12) and np.allclose(r.var(-1), 1, atol=1e-12)


# ---------------------------------------------------------------------------
# attention
def brute_attention(q, k, v, n_heads):
    T, d = q.shape
    S = k.shape[0]
    dh = d // n_heads
    out = [[0.0] * d for _ in range(T)]
    for h in range(n_heads):
        for i in range(T):
            last = S - T + i
            sc = []
            for j in range(last + 1):
                sc.append(sum(q[i][h * dh + c] * k[j][h * dh + c] for c in range(dh)))
            m = max(sc)
            e = [math.exp(s - m) for s in sc]
            z = sum(e)
            for c in range(dh):
                out[i][h * dh + c] = sum(e[j] / z * v[j][h * dh + c] for j in range(last + 1))
    return np.array(out)


@pytest.mark.parametrize("T,S,d,h", [(1, 1, 4, 1), (3, 3, 8, 2), (2, 5, 6, 3), (5, 5, 4, 2)])
def test_attention_vs_brute_force(T, S, d, h):
    rng = np.random.default_rng(T * 100 + S)
    q, k, v = (rng.standard_normal((n, d)) for n in (T, S, S))
    assert np.allclose(causal_attention(q, k, v, h), brute_attention(q, k, v, h),
                       rtol=1e-12, atol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(3)
    d, h = 8, 2
    # one key: the output is that key's value, whatever the query
    q, k, v = rng.standard_normal((1, d)), rng.standard_normal((1, d)), rng.standard_normal((1, d))
    assert np.allclose(causal_attention(q, k, v, h), v, atol=1e-14)
    # all keys equal: uniform weights, the last query averages every value
    S = 5
    k = np.repeat(rng.standard_normal((1, d)), S, axis=0)
    v = rng.standard_normal((S, d))
    q = rng.standard_normal((S, d))
    out = causal_attention(q, k, v, h)
    for i in range(S):
        assert np.allclose(out[i], v[:i + 1].mean(0), atol=1e-13)
    # one score far above the others selects its value
    k = np.eye(S, d) * 60.0
    q = np.zeros((1, d))
    q[0, 2] = q[0, 6] = 1.0          # head 0 prefers key 2; head 1 has no key 6 -> all zero
    out = causal_attention(q, k, v, h)
    assert np.allclose(out[0, :4], v[2, :4], atol=1e-20)
    assert np.allclose(out[0, 4:], v[:, 4:].mean(0), atol=1e-13)


# ---------------------------------------------------------------------------
# hand-built models (eps = 0 throughout; values derived in the comments)
def test_embedding_offset_final_norm_tied_head():
    """All layer weights zero: layers are the identity (attention of zero
    values is zero, MLP of zero weights is zero), so the logits are
    LN_f(tok[id] + pos[p + 2]) . tok^T."""
    w = HandWeights(d=4, h=1, F=2, V=3, L=1, n_pos_rows=5)
    w.tok = np.array([[1.0, 0, 0, 0], [0, 1, 0, 0], [0, 0, 1, -1]])
    w.pos = np.array([[50.0, 0, 0, 0], [0, 50, 0, 0], [0, 0, 0, 0], [0, 0, 2, 0], [9, 9, 9, 9]])
    w.lnf_g = np.array([2.0, 1, 1, 1])
    w.lnf_b = np.array([0, 0, 0, 0.5])
    logits = OracleDecoder(w, np.float64).forward(np.array([[0, 1]]))[0]
    # p=0: x = [1,0,0,0], mean 1/4, var 3/16 -> LN = [3, -1, -1, -1]/sqrt(3)
    #      gamma/beta -> [2*sqrt3, -1/sqrt3, -1/sqrt3, -1/sqrt3 + 0.5]
    r3 = math.sqrt(3)
    assert np.allclose(logits[0], [2 * r3, -1 / r3, -1 / r3 - (-1 / r3 + 0.5)], atol=1e-14)
    # p=1: x = [0,1,2,0], mean 3/4, var 11/16 -> LN = [-3, 1, 5, -3]/sqrt(11)
    r11 = math.sqrt(11)
    ln = np.array([-6 / r11, 1 / r11, 5 / r11, -3 / r11 + 0.5])
    assert np.allclose(logits[1], [ln[0], ln[1], ln[2] - ln[3]], atol=1e-14)


def test_uniform_attention_residual_and_causal_mask():
    """Wq = Wk = 0 gives equal scores, so position i averages the values of
    positions 0..i; Wv = Wo = I makes the values the LN1 outputs."""
    w = HandWeights(d=4, h=2, F=2, V=3, L=1, n_pos_rows=5)
    L = w.layers[0]
    L["wqkv"][8:12] = np.eye(4)
    L["wo"] = np.eye(4)
    x0 = np.array([[1.0, 0, 0, 0], [0, 1, 2, 0]])
    u0 = np.array([3.0, -1, -1, -1]) / math.sqrt(3)          # LN(x0[0])
    u1 = np.array([-3.0, 1, 5, -3]) / math.sqrt(11)          # LN(x0[1])
    dec = OracleDecoder(w, np.float64)
    x1, k, v = dec.layer_forward(dec.layer(0), x0, None, None)
    assert np.allclose(x1[0], x0[0] + u0, atol=1e-14)
    assert np.allclose(x1[1], x0[1] + (u0 + u1) / 2, atol=1e-14)
    assert np.allclose(v, [u0, u1], atol=1e-14) and np.allclose(k, 0)


def test_query_scaling_and_bias():
    """One head of width 4 (scale 1/2); Wq = Wk = I, bq = [0,0,0,2]: query
    position 1 scores key j with (u1 + bq) . u_j / 2."""
    w = HandWeights(d=4, h=1, F=2, V=3, L=1, n_pos_rows=5)
    L = w.layers[0]
    L["wqkv"][0:4] = np.eye(4)
    L["wqkv"][4:8] = np.eye(4)
    L["wqkv"][8:12] = np.eye(4)
    L["bqkv"][3] = 2.0
    x0 = np.array([[1.0, 0, 0, 0], [0, 1, 2, 0]])
    u0 = np.array([3.0, -1, -1, -1]) / math.sqrt(3)
    u1 = np.array([-3.0, 1, 5, -3]) / math.sqrt(11)
    qv = u1 + np.array([0, 0, 0, 2.0])
    s0, s1 = qv @ u0 / 2, qv @ u1 / 2
    p0 = math.exp(s0) / (math.exp(s0) + math.exp(s1))
    dec = OracleDecoder(w, np.float64)
    x1, _, _ = dec.layer_forward(dec.layer(0), x0, None, None)
    # Wo = 0: the attention output does not reach x; check it through Wo = I
    assert np.allclose(x1, x0, atol=1e-15)
    L["wo"] = np.eye(4)
    x1, _, _ = dec.layer_forward(dec.layer(0), x0, None, None)
    assert np.allclose(x1[1], x0[1] + p0 * u0 + (1 - p0) * u1, atol=1e-14)
    assert np.allclose(x1[0], x0[0] + u0, atol=1e-14)


def test_relu_mlp_on_second_norm():
    """Attention off; MLP h = relu(W1 a + b1) with W1 = [e0; -e0], b1 = [-1, 0],
    W2 sums both units into coordinate 0, b2 = [0, 0, 0, 0.25]."""
    w = HandWeights(d=4, h=1, F=2, V=3, L=1, n_pos_rows=5)
    L = w.layers[0]
    L["w1"] = np.array([[1.0, 0, 0, 0], [-1.0, 0, 0, 0]])
    L["b1"] = np.array([-1.0, 0])
    L["w2"] = np.array([[1.0, 1], [0, 0], [0, 0], [0, 0]])
    L["b2"] = np.array([0, 0, 0, 0.25])
    L["ln2_g"] = np.array([2.0, 1, 1, 1])
    x0 = np.array([[1.0, 0, 0, 0], [0, 1, 2, 0]])
    a0 = 2 * 3 / math.sqrt(3)            # 2 * LN(x0[0])[0]
    a1 = 2 * -3 / math.sqrt(11)          # 2 * LN(x0[1])[0]
    dec = OracleDecoder(w, np.float64)
    x1, _, _ = dec.layer_forward(dec.layer(0), x0, None, None)
    assert np.allclose(x1[0], x0[0] + [max(a0 - 1, 0) + max(-a0, 0), 0, 0, 0.25], atol=1e-14)
    assert np.allclose(x1[1], x0[1] + [max(a1 - 1, 0) + max(-a1, 0), 0, 0, 0.25], atol=1e-14)


# ---------------------------------------------------------------------------
# whole-decoder brute force and invariants
def brute_decoder(w, tokens, fp16_act=False):
    """Scalar-loop forward of one sequence (float64, math only); with fp16_act
    the LayerNorm outputs, q, k, v, attention output and FC1 output are
    rounded to fp16."""
    s = w.shape
    d, H, F = s.d_model, s.n_heads, s.d_ffn
    dh = d // H
    T = len(tokens)

    def r(vec):
        return [float(np.float16(a)) for a in vec] if fp16_act else vec

    def ln(vec, g, b):
        mu = sum(vec) / d
        var = sum((a - mu) ** 2 for a in vec) / d
        return [(vec[c] - mu) / math.sqrt(var + s.ln_eps) * g[c] + b[c] for c in range(d)]

    def lin(W, bias, vec):
        return [sum(W[r][c] * vec[c] for c in range(len(vec))) + bias[r] for r in range(len(W))]

    xs = [[w.tok[tokens[p]][c] + w.pos[p + s.pos_offset][c] for c in range(d)] for p in range(T)]
    for L in w.layers:
        qkv = [lin(L["wqkv"], L["bqkv"], r(ln(x, L["ln1_g"], L["ln1_b"]))) for x in xs]
        qs = [r([a / math.sqrt(dh) for a in row[:d]]) for row in qkv]
        ks = [r(row[d:2 * d]) for row in qkv]
        vs = [r(row[2 * d:]) for row in qkv]
        new = []
        for i in range(T):
            o = [0.0] * d
            for hh in range(H):
                sc = [sum(qs[i][hh * dh + c] * ks[j][hh * dh + c] for c in range(dh))
                      for j in range(i + 1)]
                m = max(sc)
                e = [math.exp(a - m) for a in sc]
                for c in range(dh):
                    o[hh * dh + c] = sum(e[j] * vs[j][hh * dh + c] for j in range(i + 1)) / sum(e)
            x = [xs[i][c] + v for c, v in enumerate(lin(L["wo"], L["bo"], r(o)))]
            hid = r([max(a, 0.0) for a in lin(L["w1"], L["b1"], r(ln(x, L["ln2_g"], L["ln2_b"])))])
            new.append([x[c] + v for c, v in enumerate(lin(L["w2"], L["b2"], hid))])
        xs = new
    out = []
    for x in xs:
        y = r(ln(x, w.lnf_g, w.lnf_b))
        out.append([sum(w.tok[t][c] * y[c] for c in range(d)) for t in range(s.vocab)])
    return np.array(out)


def test_decoder_vs_scalar_brute_force():
    w = random_hand()
    toks = np.array([[3, 1, 4, 1, 5], [9, 2, 6, 5, 3]])
    got = OracleDecoder(w, np.float64).forward(toks)
    for b in range(2):
        assert np.allclose(got[b], brute_decoder(w, list(toks[b])), rtol=1e-11, atol=1e-11)


def test_fp16_activation_mode_vs_scalar_brute_force():
    """The fp16-activation reading against the scalar decoder that rounds
    the same tensors, and its distance from the all-float64 decoder."""
    w = random_hand(d=16, h=2, F=24, seed=31)
    toks = np.array([[3, 1, 4, 1, 5, 9]])
    got = OracleDecoder(w, np.float64, fp16_operands=True).forward(toks)[0]
    assert np.allclose(got, brute_decoder(w, list(toks[0]), fp16_act=True), rtol=1e-11, atol=1e-11)
    exact = OracleDecoder(w, np.float64).forward(toks)[0]
    rel = np.abs(got - exact).max() / np.abs(exact).max()
    assert 0 < rel < 1e-2


def test_incremental_decode_equals_full_recompute():
    w = random_hand(seed=5)
    toks = np.array([[1, 2, 3, 4, 5, 6, 7], [7, 6, 5, 4, 3, 2, 1], [0, 0, 10, 0, 0, 10, 0]])
    dec = OracleDecoder(w, np.float64)
    full = dec.forward(toks)
    P = 3
    logits, cache = dec.prefill(toks[:, :P])
    assert np.allclose(logits, full[:, P - 1], rtol=1e-12, atol=1e-12)
    for t in range(P, toks.shape[1]):
        step = dec.decode(cache, toks[:, t])
        assert np.allclose(step, full[:, t], rtol=1e-12, atol=1e-12)


def test_forward_last_positions_are_the_full_pass_tail():
    """forward(last=n) applies the head to the last n positions only: the
    same values as the tail of the full pass (OPT and LLaMA oracles)."""
    w = random_hand(seed=5)
    toks = np.array([[1, 2, 3, 4, 5, 6, 7], [7, 6, 5, 4, 3, 2, 1]])
    dec = OracleDecoder(w, np.float64)
    full = dec.forward(toks)
    # equal up to the summation order of the head's matrix product (fp64)
    for n in (1, 3, 7):
        assert np.allclose(dec.forward(toks, last=n), full[:, -n:], rtol=1e-12, atol=1e-12)
    shape = synth.LlamaShape(2, 64, 4, 2, 96, vocab=50, max_pos=16)
    ld = decoder_for(synth.SyntheticLlama(shape, seed=3, gain_std=0.2), np.float64)
    lt = np.array([[3, 1, 4, 1, 5, 9]])
    assert np.allclose(ld.forward(lt, last=2), ld.forward(lt)[:, -2:], rtol=1e-12, atol=1e-12)
    assert np.allclose(ld.forward(lt, layers=1, last=4), ld.forward(lt, layers=1)[:, -4:],
                       rtol=1e-12, atol=1e-12)


def test_causality_and_batch_independence():
    w = random_hand(seed=6)
    toks = np.array([[1, 2, 3, 4, 5, 6], [6, 5, 4, 3, 2, 1]])
    dec = OracleDecoder(w, np.float64)
    base = dec.forward(toks)
    pert = toks.copy()
    pert[0, 3] = 9
    out = dec.forward(pert)
    assert np.allclose(out[0, :3], base[0, :3], rtol=0, atol=0)
    assert not np.allclose(out[0, 3:], base[0, 3:])
    assert np.array_equal(out[1], base[1])
    swapped = dec.forward(toks[::-1])
    assert np.allclose(swapped[::-1], base, rtol=0, atol=0)


def test_float32_close_to_float64():
    w = random_hand(seed=8)
    toks = np.array([[1, 2, 3, 4]])
    a = OracleDecoder(w, np.float64).forward(toks)
    b = OracleDecoder(w, np.float32).forward(toks)
    assert b.dtype == np.float32
    assert np.abs(a - b).max() / np.abs(a).max() < 1e-5


def test_greedy_ties_lowest_index():
    logits = np.array([[0.5, 2.0, 2.0, -1.0], [3.0, 3.0, 3.0, 3.0], [-1, -2, -0.5, -0.5]])
    assert OracleDecoder.argmax(logits).tolist() == [1, 0, 2]


# ---------------------------------------------------------------------------
# int4
def test_int4_nibble_order_and_dequant_hand():
    # one row, 64 inputs: byte i holds code(2i) low, code(2i+1) high
    q = np.zeros((1, 32), dtype=np.uint8)
    q[0, 0] = 0x21      # code0 = 1, code1 = 2
    q[0, 31] = 0xF0     # code62 = 0, code63 = 15
    sm = np.array([[[0.5, -1.0]]], dtype=np.float16)     # scale 0.5, min -1
    w = dequant_int4_g64(q, sm, np.float64)
    assert w.shape == (1, 64)
    assert w[0, 0] == 1 * 0.5 - 1 and w[0, 1] == 2 * 0.5 - 1
    assert w[0, 62] == -1.0 and w[0, 63] == 15 * 0.5 - 1
    assert (w[0, 2:62] == -1.0).all()
    # groups are per 64 inputs and per row
    q2 = np.full((2, 64), 0x11, dtype=np.uint8)
    sm2 = np.array([[[1, 0], [2, 0]], [[0.25, 1], [0, 3]]], dtype=np.float16)
    w2 = dequant_int4_g64(q2, sm2, np.float64)
    assert (w2[0, :64] == 1).all() and (w2[0, 64:] == 2).all()
    assert (w2[1, :64] == 1.25).all() and (w2[1, 64:] == 3).all()


def test_int4_roundtrip_error_bound():
    w16 = synth.normal_f16(4, 4, 64 * 512).reshape(64, 512)
    q, sm = synth.quant_int4_g64(w16)
    deq = dequant_int4_g64(q, sm, np.float64)
    s = sm[..., 0].astype(np.float64).repeat(64, axis=1)
    m = sm[..., 1].astype(np.float64).repeat(64, axis=1)
    w = w16.astype(np.float64)
    # inside the code range the error is at most half a step; at the top end
    # the fp16-rounded scale can leave up to 15 * |scale - scale16| + |min - min16|
    mx = w.reshape(64, 8, 64).max(-1).repeat(64, axis=1)
    mn = w.reshape(64, 8, 64).min(-1).repeat(64, axis=1)
    slack = 15 * np.abs((mx - mn) / 15 - s) + np.abs(mn - m)
    assert (np.abs(deq - w) <= s / 2 + slack + 1e-12).all()
    # values on an exactly representable grid (step 1/64, min -1/8) come back exactly
    grid = np.tile((np.arange(64) % 16) / 64.0 - 0.125, (3, 1))
    qg, smg = synth.quant_int4_g64(grid.astype(np.float16))
    assert (dequant_int4_g64(qg, smg, np.float64) == grid).all()


def test_int4_weights_drive_the_same_decoder():
    shape = synth.OPTShape(2, 64, 4, 256, vocab=97, max_pos=16)
    m16 = synth.SyntheticOPT(shape, seed=3)
    m4 = synth.SyntheticOPT(shape, seed=3, wfmt="int4")
    toks = np.array([[1, 5, 9, 13]])
    a = OracleDecoder(m16, np.float64).forward(toks)
    b = OracleDecoder(m4, np.float64).forward(toks)
    # int4 codes move every weight by at most ~half a step (~0.004 here)
    assert not np.allclose(a, b, atol=1e-6)
    assert np.abs(a - b).max() < 0.25 * np.abs(a).max()


def test_fp16_operands_expand_int4_weights_to_fp16():
    """In the fp16-operand reading an INT4 model computes exactly as the fp16
    model whose weights are the expanded codes rounded to fp16."""
    shape = synth.OPTShape(2, 64, 4, 256, vocab=97, max_pos=16)
    m4 = synth.SyntheticOPT(shape, seed=3, wfmt="int4")

    class Expanded:
        def __init__(self):
            self.shape, self.wfmt = m4.shape, "fp16"

        def layer(self, j):
            out = dict(m4.layer(j))
            for nm in ("wqkv", "wo", "w1", "w2"):
                out[nm] = dequant_int4_g64(*out[nm], np.float64).astype(np.float16)
            return out

        def tok_emb(self):
            return m4.tok_emb()

        def pos_emb(self):
            return m4.pos_emb()

        def lnf(self):
            return m4.lnf()

    toks = np.array([[1, 5, 9, 13]])
    a = OracleDecoder(m4, np.float64, fp16_operands=True).forward(toks)
    b = OracleDecoder(Expanded(), np.float64, fp16_operands=True).forward(toks)
    assert np.array_equal(a, b)
    assert not np.array_equal(a, OracleDecoder(m4, np.float64).forward(toks))


# ---------------------------------------------------------------------------
# shapes and bytes
def test_parameter_counts_of_opt_shapes():
    # OPT-125m: 50272*768 + 2050*768 + 12*(12*768^2 + 13*768) + 2*768
    assert param_count(12, 768, 3072, 50272, 2050) == 125_239_296
    assert round(param_count(32, 4096, 16384, 50272, 2050) / 1e9, 2) == 6.66
    assert round(param_count(40, 5120, 20480, 50272, 2050) / 1e9, 2) == 12.85
    assert round(param_count(48, 7168, 28672, 50272, 2050) / 1e9, 2) == 29.97


def test_weight_bytes_against_paper_statements():
    with open(os.path.join(GOLDEN, "paper_weight_sizes.json")) as f:
        facts = json.load(f)
    opt67 = facts["opt_6_7b_fp16_weight_gb"]
    gb = 2 * param_count(32, 4096, 16384, 50272, 2050) / 1e9
    assert abs(gb - opt67["value"]) <= opt67["tolerance"]
    big = facts["30b_fp16_weight_gb_at_least"]
    assert 2 * param_count(48, 7168, 28672, 50272, 2050) / 1e9 >= big["value"]


def test_streamed_bytes_per_step_closed_forms():
    for d in (768, 4096, 5120, 7168):
        F = 4 * d
        fp16_layer = streamed_bytes_per_step(1, d, F, 50272, "fp16", stream_head=False)
        assert fp16_layer == 2 * (12 * d * d + 13 * d)
        int4_layer = streamed_bytes_per_step(1, d, F, 50272, "int4", stream_head=False)
        assert int4_layer == 0.5625 * 12 * d * d + 26 * d
    # OPT-6.7B, fp16, 32 layers plus the tied head: 13.30 GB per step
    assert round(streamed_bytes_per_step(32, 4096, 16384, 50272, "fp16") / 1e9, 2) == 13.30
    # KV prefix in host memory: 2 (K, V) * b * t * d * 2 bytes per layer
    kv = streamed_bytes_per_step(2, 64, 256, 10, "fp16", stream_head=False, kv_batch=3, kv_len=5)
    assert kv - streamed_bytes_per_step(2, 64, 256, 10, "fp16", stream_head=False) == \
        2 * 2 * 3 * 5 * 64 * 2
    # the same prefix as INT4 rows: d/2 code bytes and d/64 (scale, min) pairs
    kv4 = streamed_bytes_per_step(2, 64, 256, 10, "fp16", stream_head=False, kv_batch=3, kv_len=5,
                                  kv_fmt="int4")
    assert kv4 - streamed_bytes_per_step(2, 64, 256, 10, "fp16", stream_head=False) == \
        2 * 2 * 3 * 5 * (32 + 4)


# ---------------------------------------------------------------------------
# INT4 KV cache entries
def test_kv_int4_grid_values_are_exact():
    """Rows built as m + code * s (fp16-exact, each group holding codes 0 and
    15) come back with exactly those codes, s and m, and dequantize exactly."""
    rng = np.random.default_rng(21)
    R, d = 5, 256
    codes = rng.integers(0, 16, (R, d))
    codes[:, 0::64] = 0
    codes[:, 1::64] = 15
    s = (2.0 ** rng.integers(-8, 0, (R, d // 64))).astype(np.float16)
    m = (rng.integers(-64, 64, (R, d // 64)) / 64.0).astype(np.float16)
    x = m.astype(np.float64).repeat(64, 1) + codes * s.astype(np.float64).repeat(64, 1)
    assert np.array_equal(x.astype(np.float16).astype(np.float64), x)
    q, sm = quant_kv_int4_g64(x.astype(np.float16))
    assert np.array_equal(sm[..., 0], s) and np.array_equal(sm[..., 1], m)
    assert np.array_equal(q & 0x0F, codes[:, 0::2]) and np.array_equal(q >> 4, codes[:, 1::2])
    assert np.array_equal(dequant_int4_g64(q, sm, np.float64), x)


def test_kv_int4_rounding_half_even_and_nibbles():
    """Group with min 0 and max 15 (scale exactly 1): halves round to even,
    and codes pack two per byte, even element low."""
    row = np.zeros(64, np.float16)
    row[:8] = [0, 15, 0.5, 1.5, 2.5, 14.5, 7.25, 7.75]
    q, sm = quant_kv_int4_g64(row[None])
    assert sm[0, 0, 0] == 1 and sm[0, 0, 1] == 0
    assert list(q[0, :4]) == [0 | 15 << 4, 0 | 2 << 4, 2 | 14 << 4, 7 | 8 << 4]
    ramp = np.arange(16, dtype=np.float16).repeat(4)          # codes 0,0,0,0,1,1,1,1,...
    q, _ = quant_kv_int4_g64(ramp[None])
    assert list(q[0, :4]) == [0x00, 0x00, 0x11, 0x11]


def test_kv_int4_roundtrip_bound_monotone_constant_groups():
    rng = np.random.default_rng(22)
    for scale in (1e-3, 0.02, 1.0, 300.0):
        x = (rng.standard_normal((7, 512)) * scale).astype(np.float16)
        x[3, 64:128] = np.float16(0.375)                      # a constant group
        q, sm = quant_kv_int4_g64(x)
        back = dequant_int4_g64(q, sm, np.float64)
        s = sm[..., 0].astype(np.float64).repeat(64, 1)
        # nearest grid point: half a step, plus fp32 rounding of the division
        err = np.abs(back - x.astype(np.float64))
        assert (err <= 0.5 * s * (1 + 1e-6) + 1e-30).all()
        assert np.array_equal(back[3, 64:128], x[3, 64:128].astype(np.float64))
        c = np.empty(x.shape, np.int64)
        c[:, 0::2], c[:, 1::2] = q & 0x0F, q >> 4
        for r in range(x.shape[0]):
            for g in range(x.shape[1] // 64):
                xs, cs = x[r, 64 * g:64 * g + 64], c[r, 64 * g:64 * g + 64]
                order = np.argsort(xs, kind="stable")
                assert (np.diff(cs[order]) >= 0).all()       # codes never decrease with x


@pytest.mark.parametrize("fp16_act", [False, True])
def test_kv_int4_incremental_decode_equals_full_recompute(fp16_act):
    w = random_hand(d=64, h=2, F=32, seed=23)
    toks = np.array([[1, 2, 3, 4, 5, 6, 7], [7, 6, 5, 4, 3, 2, 1]])
    dec = OracleDecoder(w, np.float64, kv_int4=True, fp16_operands=fp16_act)
    full = dec.forward(toks)
    assert not np.allclose(full, OracleDecoder(w, np.float64).forward(toks), rtol=1e-6)
    P = 3
    logits, cache = dec.prefill(toks[:, :P])
    assert np.allclose(logits, full[:, P - 1], rtol=1e-12, atol=1e-12)
    for t in range(P, toks.shape[1]):
        assert np.allclose(dec.decode(cache, toks[:, t]), full[:, t], rtol=1e-12, atol=1e-12)


def test_kv_int4_values_are_the_cached_entries():
    """With Wk = Wv = 0 every key and value row is its bias, so the INT4-cache
    decoder must equal the plain decoder whose biases are replaced by their
    cache entries (and differ from the plain one with the original biases)."""
    w = random_hand(d=64, h=2, F=32, seed=24)
    for lw in w.layers:
        lw["wqkv"][64:] = 0
    toks = np.array([[1, 2, 3, 4, 5]])
    got = OracleDecoder(w, np.float64, kv_int4=True).forward(toks)
    plain = OracleDecoder(w, np.float64).forward(toks)
    assert not np.allclose(got, plain, rtol=1e-9)
    for lw in w.layers:
        kv = lw["bqkv"][64:].reshape(2, 64).astype(np.float16)
        q, sm = quant_kv_int4_g64(kv)
        lw["bqkv"] = np.concatenate([lw["bqkv"][:64], dequant_int4_g64(q, sm, np.float64).ravel()])
    assert np.allclose(got, OracleDecoder(w, np.float64).forward(toks), rtol=1e-12, atol=1e-12)
