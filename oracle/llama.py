"""Plain, slow, obviously correct LLaMA-3.1-style decoder on the CPU (numpy).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and ``bench.py``'s ``cpu_baseline`` leg; never by the GPU library.

The paper evaluates LLaMA3.1 (8B, 70B) beside OPT (Section 4.1) and writes
its memory model for that family (Section 3.5): grouped-query attention
with h heads and h_kv key/value heads, an MLP of hidden width d_h with three
matrices, an input embedding and an output head of d x V each.  It does not
restate the architecture; the readings here are those of the published
LLaMA 3.1 models:

* pre-norm blocks with RMSNorm (x / sqrt(mean(x^2) + eps) * g), eps 1e-5,
  and a final RMSNorm;
* q, k, v projections without biases; rotary positions on q and k, pairing
  element i with element i + head_dim/2 of every head, angle p * w_i with
  w_i = theta^(-2i/head_dim), theta 500000, and the 3.1 frequency scaling
  (wavelengths longer than orig/low_freq_factor divided by `factor`, shorter
  than orig/high_freq_factor kept, a linear blend in between);
* query head j reads key/value head j // (h / h_kv); q is scaled by
  head_dim**-0.5 (as in the OPT oracle; the rotation is linear, so the
  order of scaling and rotating does not matter), causal softmax;
* SwiGLU MLP: down(silu(gate(x)) * up(x)), gate and up stacked in one
  [2 d_ffn][d] matrix (gate rows first);
* untied output head, no biases anywhere.

INT4 weights and the INT4 KV cache use the OPT oracle's encodings
(``dequant_int4_g64``, ``quant_kv_int4_g64``); keys enter the cache after
their rotation.  ``fp16_operands`` rounds the tensors the kernels hold in
fp16 (norm outputs, q, k, v after rotation, attention output, SwiGLU output,
expanded INT4 weights).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

import numpy as np

from .opt import MATRICES, dequant_int4_g64, quant_kv_int4_g64


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * g


def rope_frequencies(head_dim: int, theta: float, factor: float = 0.0,
                     low_freq_factor: float = 1.0, high_freq_factor: float = 4.0,
                     orig_max_pos: int = 8192) -> np.ndarray:
    """w_i = theta^(-2i/head_dim), i < head_dim/2, in float64, with the 3.1
    scaling when factor > 0: a component whose wavelength 2 pi / w exceeds
    orig/low_freq_factor is divided by factor; one shorter than
    orig/high_freq_factor is kept; in between w' = (1 - s) w / factor + s w
    with s = (orig / wavelength - low_freq_factor) / (high - low)."""
    w = theta ** (-np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)
    if factor <= 0:
        return w
    wavelen = 2 * np.pi / w
    long_limit = orig_max_pos / low_freq_factor
    short_limit = orig_max_pos / high_freq_factor
    s = (orig_max_pos / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    blended = (1 - s) * w / factor + s * w
    return np.where(wavelen > long_limit, w / factor,
                    np.where(wavelen < short_limit, w, blended))


def apply_rope(x: np.ndarray, positions: np.ndarray, freqs: np.ndarray) -> np.ndarray:
    """Rotate every head of x [T][n_heads * head_dim]: the pair (i, i + half)
    of position p turns by the angle p * freqs[i]."""
    T, width = x.shape
    half = freqs.shape[0]
    hd = 2 * half
    ang = positions.astype(np.float64)[:, None] * freqs[None, :]       # [T][half]
    c = np.cos(ang).astype(x.dtype)[:, None, :]
    s = np.sin(ang).astype(x.dtype)[:, None, :]
    xh = x.reshape(T, width // hd, hd)
    a, b = xh[..., :half], xh[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1).reshape(T, width)


def swiglu(gate: np.ndarray, up: np.ndarray) -> np.ndarray:
    """silu(gate) * up with silu(g) = g / (1 + exp(-g))."""
    return gate / (1 + np.exp(-gate)) * up


def gqa_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int,
                  n_kv_heads: int) -> np.ndarray:
    """T queries [T][h*dh] (already scaled) over S >= T keys and values
    [S][h_kv*dh]; query i sits at position S - T + i; head j uses key/value
    head j // (h / h_kv).  Softmax is max-subtracted."""
    T, d = q.shape
    S = k.shape[0]
    dh = d // n_heads
    group = n_heads // n_kv_heads
    out = np.empty_like(q)
    mask = np.arange(S)[None, :] <= (S - T + np.arange(T))[:, None]
    for j in range(n_heads):
        kj = k[:, (j // group) * dh:(j // group + 1) * dh]
        vj = v[:, (j // group) * dh:(j // group + 1) * dh]
        sc = q[:, j * dh:(j + 1) * dh] @ kj.T
        sc = np.where(mask, sc, -np.inf)
        p = np.exp(sc - sc.max(axis=-1, keepdims=True))
        p = p / p.sum(axis=-1, keepdims=True)
        out[:, j * dh:(j + 1) * dh] = p @ vj
    return out


def llama_param_count(n_layers: int, d: int, n_heads: int, n_kv_heads: int, d_ffn: int,
                      vocab: int) -> int:
    """Section 3.5's count in elements: 2 W_embed + l (W_mha + W_mlp) with
    W_mha = d (2d + 2d h_kv/h + 1) (the form of Appendix B), W_mlp =
    d (3 d_h + 1), plus the final norm."""
    mha = d * (2 * d + 2 * d * n_kv_heads // n_heads + 1)
    mlp = d * (3 * d_ffn + 1)
    return 2 * d * vocab + n_layers * (mha + mlp) + d


def llama_kv_bytes(n_layers: int, d: int, n_heads: int, n_kv_heads: int, batch: int,
                   seq: int, p: int = 2) -> int:
    """Section 3.5's KV cache size C = 2 p b s l d h_kv / h."""
    return 2 * p * batch * seq * n_layers * d * n_kv_heads // n_heads


class LlamaDecoder:
    """The LLaMA-3.1-style forward pass over a weight provider.

    ``weights`` provides ``shape`` (n_layers, d_model, n_heads, n_kv_heads,
    d_ffn, vocab, ln_eps and the rope fields), ``wfmt``, ``tok_emb()``,
    ``lm_head()``, ``lnf()`` -> (g, None) and ``layer(j)`` -> dict with
    ln1_g, wqkv, wo, ln2_g, w1 (gate and up stacked), w2 (int4 matrices as
    (codes, scale_min) pairs).  Same interface as OracleDecoder.
    """

    def __init__(self, weights, dtype=np.float32, kv_int4: bool = False,
                 fp16_operands: bool = False):
        self.w = weights
        self.s = weights.shape
        self.dtype = dtype
        self.kv_int4 = kv_int4
        self.fp16_operands = fp16_operands
        s = self.s
        self.freqs = rope_frequencies(s.head_dim, s.rope_theta, s.rope_factor,
                                      s.rope_low_freq_factor, s.rope_high_freq_factor,
                                      s.rope_orig_max_pos)
        self._tok = self._head = self._lnf = None

    def _f(self, a) -> np.ndarray:
        return np.asarray(a).astype(self.dtype)

    def act(self, a: np.ndarray) -> np.ndarray:
        if not self.fp16_operands:
            return a
        return a.astype(np.float16).astype(self.dtype)

    def kv_entry(self, a: np.ndarray) -> np.ndarray:
        if not self.kv_int4:
            return a
        codes, sm = quant_kv_int4_g64(a.astype(np.float16))
        return dequant_int4_g64(codes, sm, self.dtype)

    def tok_emb(self) -> np.ndarray:
        if self._tok is None:
            self._tok = self._f(self.w.tok_emb())
        return self._tok

    def lm_head(self) -> np.ndarray:
        if self._head is None:
            self._head = self._f(self.w.lm_head())
        return self._head

    def lnf(self) -> np.ndarray:
        if self._lnf is None:
            self._lnf = self._f(self.w.lnf()[0])
        return self._lnf

    def layer(self, j: int) -> Dict[str, np.ndarray]:
        out = {}
        for name, val in self.w.layer(j).items():
            if name in MATRICES and self.w.wfmt == "int4":
                out[name] = self.act(dequant_int4_g64(val[0], val[1], self.dtype))
            else:
                out[name] = self._f(val)
        return out

    def embed(self, tokens: np.ndarray) -> np.ndarray:
        return self.tok_emb()[tokens]

    def layer_forward(self, L: Dict[str, np.ndarray], x: np.ndarray, positions: np.ndarray,
                      past_k: Optional[np.ndarray], past_v: Optional[np.ndarray]):
        """One layer on one sequence: x [T][d] at `positions`; past keys and
        values [S0][h_kv*dh] (already rotated / cached) or None."""
        s = self.s
        d, h, hkv, dh = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim
        a = self.act(rms_norm(x, L["ln1_g"], s.ln_eps))
        qkv = a @ L["wqkv"].T
        q = self.act(apply_rope(qkv[:, :h * dh] * (dh ** -0.5), positions, self.freqs))
        k = self.kv_entry(self.act(apply_rope(qkv[:, h * dh:(h + hkv) * dh], positions,
                                              self.freqs)))
        v = self.kv_entry(self.act(qkv[:, (h + hkv) * dh:]))
        if past_k is not None:
            k = np.concatenate([past_k, k], axis=0)
            v = np.concatenate([past_v, v], axis=0)
        o = self.act(gqa_attention(q, k, v, h, hkv))
        x = x + o @ L["wo"].T
        a2 = self.act(rms_norm(x, L["ln2_g"], s.ln_eps))
        gu = a2 @ L["w1"].T
        F = s.d_ffn
        gate, up = gu[:, :F], gu[:, F:]
        hdn = self.act(swiglu(gate, up))
        x = x + hdn @ L["w2"].T
        return x, k, v

    def head(self, x: np.ndarray) -> np.ndarray:
        return self.act(rms_norm(x, self.lnf(), self.s.ln_eps)) @ self.lm_head().T

    def forward(self, tokens: np.ndarray, layers: Optional[int] = None,
                last: Optional[int] = None) -> np.ndarray:
        """Full recomputation: logits [b][s][V] (or of the last ``last``
        positions only, [b][last][V])."""
        tokens = np.asarray(tokens)
        B, S = tokens.shape
        nl = self.s.n_layers if layers is None else layers
        first = 0 if last is None else S - last
        pos = np.arange(S)
        xs = [self.embed(tokens[i]) for i in range(B)]
        for j in range(nl):
            L = self.layer(j)
            xs = [self.layer_forward(L, x, pos, None, None)[0] for x in xs]
        return np.stack([self.head(x[first:]) for x in xs])

    def prefill(self, tokens: np.ndarray) -> Tuple[np.ndarray, List]:
        tokens = np.asarray(tokens)
        B, P = tokens.shape
        pos = np.arange(P)
        xs = [self.embed(tokens[i]) for i in range(B)]
        cache = []
        for j in range(self.s.n_layers):
            L = self.layer(j)
            kv = []
            for i in range(B):
                xs[i], k, v = self.layer_forward(L, xs[i], pos, None, None)
                kv.append((k, v))
            cache.append(kv)
        return np.stack([self.head(x[-1:])[0] for x in xs]), cache

    def decode(self, cache: List, tokens: np.ndarray) -> np.ndarray:
        tokens = np.asarray(tokens)
        B = tokens.shape[0]
        t = cache[0][0][0].shape[0]
        xs = [self.embed(tokens[i:i + 1]) for i in range(B)]
        for j in range(self.s.n_layers):
            L = self.layer(j)
            for i in range(B):
                pk, pv = cache[j][i]
                xs[i], k, v = self.layer_forward(L, xs[i], np.array([t]), pk, pv)
                cache[j][i] = (k, v)
        return np.stack([self.head(x)[0] for x in xs])

    @staticmethod
    def argmax(logits: np.ndarray) -> np.ndarray:
        return np.argmax(logits, axis=-1).astype(np.int32)


def decoder_for(weights, *args, **kw):
    """The oracle decoder of the weights' model family."""
    from .opt import OracleDecoder
    if getattr(weights.shape, "family", "opt") == "llama":
        return LlamaDecoder(weights, *args, **kw)
    return OracleDecoder(weights, *args, **kw)
