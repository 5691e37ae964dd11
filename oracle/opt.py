"""Plain, slow, obviously correct OPT decoder on the CPU (numpy).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and ``bench.py``'s ``cpu_baseline`` leg; never by the GPU library.

What is computed, and where it comes from:

* PIPO's computation tasks are the MHA and MLP layers plus the input and
  output embeddings, run one after another (Section 3.1.2, "Computation").
  Offloading, pipelining and chunked transfer only move data; they do not
  change these results (Section 3.1.1; Section 4.1 states fp16 or INT4
  weights with fp16 activations).
* The models are OPT (Section 4.1, "Model").  The paper does not restate
  the OPT architecture, so the readings used here are:
    - pre-LayerNorm blocks with a final LayerNorm, eps 1e-5;
    - learned positions, position p read at row p + pos_offset (2 for OPT);
    - q is scaled by head_dim**-0.5 after its bias is added;
    - ReLU MLP of width d_ffn; tied output embedding, no output bias;
    - greedy decoding, ties to the lowest token id.
* INT4 weights (Section 2 and Section 3.4: weights are kept in 4 bits and
  the GEMM works on them directly): a weight is q * scale + min with one fp16
  (scale, min) pair per group of 64 consecutive inputs of a row, codes
  packed two per byte with the even input in the low nibble.  The paper
  gives no recipe; this is the one the workloads define.
* INT4 KV cache (Section 2: PIPO can keep the KV cache in 4 bits too; the
  conversion belongs to the KV loading and saving tasks, Section 3.1.2).
  The paper gives no recipe; the reading here: a new key or value row is
  rounded to fp16 (activations are fp16, Section 4.1) and quantized per
  group of 64 consecutive elements with the same asymmetric (scale, min)
  scheme (quant_kv_int4_g64), and every attention -- prefill included --
  reads the cache, i.e. the dequantized values.  A row's codes depend on
  that row alone, so incremental decoding still equals full recomputation.

The default arithmetic type is float32; tests that pin the oracle run it in
float64.  With ``fp16_operands`` every tensor the kernels hold in fp16 is
rounded to fp16 (Section 4.1: fp16 activations; an INT4 weight is expanded
to an fp16 operand): the LayerNorm outputs, q, k and v, the attention
output, the FC1 output and the expanded INT4 weights; the residual stream
and the logits stay in the arithmetic type.  INT4 KV codes are decisions
taken on k and v, so comparisons with an INT4 cache use this mode (the codes
then come from the same fp16 values up to summation order).  Everything is vectorised numpy over whole tensors, with no
blocking or fusion: a layer is LN -> QKV -> causal softmax attention ->
out-projection + residual -> LN -> FC1 -> ReLU -> FC2 + residual.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Tuple

import numpy as np

MATRICES = ("wqkv", "wo", "w1", "w2")


# ---------------------------------------------------------------------------
# building blocks
def layer_norm(x: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float) -> np.ndarray:
    """LayerNorm over the last axis: (x - mean) / sqrt(var + eps) * gamma + beta,
    with the biased (population) variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gamma + beta


def dequant_int4_g64(q: np.ndarray, sm: np.ndarray, dtype=np.float32) -> np.ndarray:
    """W[n, k] = code[n, k] * scale[n, k // 64] + min[n, k // 64].

    ``q`` is [N][K/2] uint8 with code(2i) in the low nibble and code(2i+1) in
    the high nibble; ``sm`` is [N][K/64][2] fp16 holding (scale, min).  The
    product and sum are taken in ``dtype``.
    """
    N, half = q.shape
    K = 2 * half
    codes = np.empty((N, K), dtype=dtype)
    codes[:, 0::2] = q & 0x0F
    codes[:, 1::2] = q >> 4
    scale = sm[..., 0].astype(dtype)
    mn = sm[..., 1].astype(dtype)
    w = codes.reshape(N, K // 64, 64) * scale[..., None] + mn[..., None]
    return w.reshape(N, K)


def quant_kv_int4_g64(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """INT4 cache entry of fp16 rows x [R][d] (d a multiple of 64).

    Per group of 64 consecutive elements of a row, in float32:
    mn, mx = min, max; s = fp16((mx - mn) / 15); m = fp16(mn);
    code = clamp(rint((x - m) / s), 0, 15) with rint rounding half to even,
    and code = 0 where s == 0.  Returns codes [R][d/2] uint8 (element 2i in
    the low nibble of byte i) and (s, m) pairs [R][d/64][2] fp16, the layout
    dequant_int4_g64 reads.
    """
    x = np.asarray(x, dtype=np.float16).astype(np.float32)
    R, d = x.shape
    g = x.reshape(R, d // 64, 64)
    mn = g.min(axis=-1)
    mx = g.max(axis=-1)
    s16 = ((mx - mn) / np.float32(15)).astype(np.float16)
    m16 = mn.astype(np.float16)
    s32 = s16.astype(np.float32)[..., None]
    m32 = m16.astype(np.float32)[..., None]
    with np.errstate(divide="ignore", invalid="ignore"):
        c = np.rint((g - m32) / s32)
    c = np.where(s32 == 0, np.float32(0), np.clip(c, 0, 15)).astype(np.uint8).reshape(R, d)
    codes = (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8)
    sm = np.stack([s16, m16], axis=-1)
    return codes, sm


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_heads: int) -> np.ndarray:
    """Multi-head softmax attention of T queries over S >= T keys.

    q: [T][d] (already scaled), k, v: [S][d].  Query i sits at position
    S - T + i and sees keys 0 .. S - T + i.  Softmax is max-subtracted.
    """
    T, d = q.shape
    S = k.shape[0]
    dh = d // n_heads
    out = np.empty_like(q)
    qpos = np.arange(T)[:, None] + (S - T)
    mask = np.arange(S)[None, :] > qpos                       # True = not visible
    for h in range(n_heads):
        sl = slice(h * dh, (h + 1) * dh)
        scores = q[:, sl] @ k[:, sl].T                        # [T][S]
        scores = np.where(mask, -np.inf, scores)
        scores = scores - scores.max(axis=-1, keepdims=True)
        p = np.exp(scores)
        p = p / p.sum(axis=-1, keepdims=True)
        out[:, sl] = p @ v[:, sl]
    return out


# ---------------------------------------------------------------------------
# byte and parameter accounting (OPT form of the paper's weight-size model,
# Section 3.5: an MHA block holds QKV and output projections with biases, an
# MLP block two matrices with biases, plus two LayerNorms per layer)
def layer_param_count(d: int, d_ffn: int) -> int:
    return 4 * d * d + 4 * d + 2 * d * d_ffn + d_ffn + d + 4 * d


def param_count(n_layers: int, d: int, d_ffn: int, vocab: int, n_pos_rows: int) -> int:
    """Embeddings (tied output head) + layers + final LayerNorm."""
    return vocab * d + n_pos_rows * d + n_layers * layer_param_count(d, d_ffn) + 2 * d


def streamed_bytes_per_step(n_layers: int, d: int, d_ffn: int, vocab: int, wfmt: str,
                            stream_head: bool = True, kv_batch: int = 0,
                            kv_len: int = 0, kv_fmt: str = "fp16") -> int:
    """Host-to-device bytes one decode step streams: every layer's weights,
    the tied output head, and (when the KV cache lives in host memory) each
    layer's K and V prefix of kv_len positions for kv_batch sequences, a
    row of d elements taking 2 d bytes (fp16) or d/2 + d/16 (INT4 codes and
    one (scale, min) pair per 64)."""
    mats = 4 * d * d + 2 * d * d_ffn
    small = layer_param_count(d, d_ffn) - mats
    if wfmt == "fp16":
        per_layer = 2 * (mats + small)
    elif wfmt == "int4":
        per_layer = mats // 2 + (mats // 64) * 4 + 2 * small
    else:
        raise ValueError(wfmt)
    total = n_layers * per_layer
    if stream_head:
        total += 2 * vocab * d
    row = {"fp16": 2 * d, "int4": d // 2 + d // 16}[kv_fmt]
    total += n_layers * 2 * kv_batch * kv_len * row
    return total


# ---------------------------------------------------------------------------
class OracleDecoder:
    """The decoder forward pass over a weight provider.

    ``weights`` provides ``shape`` (n_layers, d_model, n_heads, d_ffn, vocab,
    pos_offset, ln_eps), ``wfmt`` ("fp16" or "int4"), ``tok_emb()``,
    ``pos_emb()``, ``lnf()`` and ``layer(j)`` -> dict with ln1_g, ln1_b, wqkv,
    bqkv, wo, bo, ln2_g, ln2_b, w1, b1, w2, b2 (matrices [out][in]; with int4
    each matrix is a (codes, scale_min) pair).  Layers are fetched one at a
    time, so the oracle never holds more than one layer's weights.
    """

    def __init__(self, weights, dtype=np.float32, kv_int4: bool = False,
                 fp16_operands: bool = False):
        self.w = weights
        self.s = weights.shape
        self.dtype = dtype
        self.kv_int4 = kv_int4
        self.fp16_operands = fp16_operands
        self._tok = None
        self._pos = None
        self._lnf = None

    # -- parameters ---------------------------------------------------------
    def _f(self, a) -> np.ndarray:
        return np.asarray(a).astype(self.dtype)

    def tok_emb(self) -> np.ndarray:
        if self._tok is None:
            self._tok = self._f(self.w.tok_emb())
        return self._tok

    def pos_emb(self) -> np.ndarray:
        if self._pos is None:
            self._pos = self._f(self.w.pos_emb())
        return self._pos

    def lnf(self):
        if self._lnf is None:
            g, b = self.w.lnf()
            self._lnf = (self._f(g), self._f(b))
        return self._lnf

    def layer(self, j: int) -> Dict[str, np.ndarray]:
        raw = self.w.layer(j)
        out = {}
        for name, val in raw.items():
            if name in MATRICES and self.w.wfmt == "int4":
                out[name] = self.act(dequant_int4_g64(val[0], val[1], self.dtype))
            else:
                out[name] = self._f(val)
        return out

    # -- pieces -------------------------------------------------------------
    def embed(self, tokens: np.ndarray, positions: np.ndarray) -> np.ndarray:
        """x = token embedding + learned position embedding at p + offset."""
        return self.tok_emb()[tokens] + self.pos_emb()[positions + self.s.pos_offset]

    def layer_forward(self, L: Dict[str, np.ndarray], x: np.ndarray,
                      past_k: Optional[np.ndarray], past_v: Optional[np.ndarray]):
        """One pre-LN decoder layer on one sequence.

        x: [T][d] hidden states of the T newest positions; past_k/past_v:
        [S0][d] keys/values of the earlier positions (or None).  Returns the
        new x and the full key/value arrays [S0 + T][d].
        """
        d = self.s.d_model
        dh = d // self.s.n_heads
        eps = self.s.ln_eps
        a = self.act(layer_norm(x, L["ln1_g"], L["ln1_b"], eps))
        qkv = a @ L["wqkv"].T + L["bqkv"]
        q = self.act(qkv[:, :d] * (dh ** -0.5))
        k = self.kv_entry(self.act(qkv[:, d:2 * d]))
        v = self.kv_entry(self.act(qkv[:, 2 * d:]))
        if past_k is not None:
            k = np.concatenate([past_k, k], axis=0)
            v = np.concatenate([past_v, v], axis=0)
        o = self.act(causal_attention(q, k, v, self.s.n_heads))
        x = x + (o @ L["wo"].T + L["bo"])
        a2 = self.act(layer_norm(x, L["ln2_g"], L["ln2_b"], eps))
        hdn = self.act(np.maximum(a2 @ L["w1"].T + L["b1"], 0))
        x = x + (hdn @ L["w2"].T + L["b2"])
        return x, k, v

    def act(self, a: np.ndarray) -> np.ndarray:
        """A tensor as the kernels hold it (fp16 with fp16_operands)."""
        if not self.fp16_operands:
            return a
        return a.astype(np.float16).astype(self.dtype)

    def kv_entry(self, a: np.ndarray) -> np.ndarray:
        """The values the KV cache holds for new key or value rows a [T][d]:
        a itself, or with an INT4 cache the dequantized int4 entry."""
        if not self.kv_int4:
            return a
        codes, sm = quant_kv_int4_g64(a.astype(np.float16))
        return dequant_int4_g64(codes, sm, self.dtype)

    def head(self, x: np.ndarray) -> np.ndarray:
        g, b = self.lnf()
        return self.act(layer_norm(x, g, b, self.s.ln_eps)) @ self.tok_emb().T

    # -- whole passes -------------------------------------------------------
    def forward(self, tokens: np.ndarray, layers: Optional[int] = None,
                last: Optional[int] = None) -> np.ndarray:
        """Full recomputation: logits [b][s][V] of every position of every
        sequence, no cache.  ``layers`` truncates the stack (a layer slice);
        ``last`` returns only the logits of the last ``last`` positions
        ([b][last][V]; the head is applied to those positions alone)."""
        tokens = np.asarray(tokens)
        B, S = tokens.shape
        nl = self.s.n_layers if layers is None else layers
        first = 0 if last is None else S - last
        pos = np.arange(S)
        xs = [self.embed(tokens[i], pos) for i in range(B)]
        for j in range(nl):
            L = self.layer(j)
            xs = [self.layer_forward(L, x, None, None)[0] for x in xs]
        return np.stack([self.head(x[first:]) for x in xs])

    def prefill(self, tokens: np.ndarray) -> Tuple[np.ndarray, List]:
        """Logits [b][V] at the last prompt position, plus the KV cache
        (per layer, per sequence: keys and values [P][d])."""
        tokens = np.asarray(tokens)
        B, P = tokens.shape
        pos = np.arange(P)
        xs = [self.embed(tokens[i], pos) for i in range(B)]
        cache = []
        for j in range(self.s.n_layers):
            L = self.layer(j)
            kv = []
            for i in range(B):
                xs[i], k, v = self.layer_forward(L, xs[i], None, None)
                kv.append((k, v))
            cache.append(kv)
        logits = np.stack([self.head(x[-1:])[0] for x in xs])
        return logits, cache

    def decode(self, cache: List, tokens: np.ndarray) -> np.ndarray:
        """One incremental step: tokens [b] at position len(cache); appends to
        the cache in place and returns logits [b][V]."""
        tokens = np.asarray(tokens)
        B = tokens.shape[0]
        t = cache[0][0][0].shape[0]
        xs = [self.embed(tokens[i:i + 1], np.array([t])) for i in range(B)]
        for j in range(self.s.n_layers):
            L = self.layer(j)
            for i in range(B):
                pk, pv = cache[j][i]
                xs[i], k, v = self.layer_forward(L, xs[i], pk, pv)
                cache[j][i] = (k, v)
        return np.stack([self.head(x)[0] for x in xs])

    @staticmethod
    def argmax(logits: np.ndarray) -> np.ndarray:
        """Greedy token: the largest logit, ties to the lowest id."""
        return np.argmax(logits, axis=-1).astype(np.int32)
