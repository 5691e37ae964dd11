"""Host-side setup around the C ABI: weights laid out in pinned host memory
for streaming, and a small Decoder wrapper over pipo_create / pipo_prefill /
pipo_decode_step.  Nothing here computes any part of the decoder.

Host layout (data merging, Section 3.3 of the paper): each layer's four
matrices -- fp16, or INT4 codes each followed by its (scale, min) pairs --
share one pinned region at 4 KiB-aligned offsets, so the copy engine streams
them without staging; the output head (the token table for OPT, the untied
head for LLaMA) has a pinned region of its own.
"""
from __future__ import annotations

import ctypes
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import binding as B

MATRIX_SHAPES = ("wqkv", "wo", "w1", "w2")
SMALL = ("ln1_g", "ln1_b", "bqkv", "bo", "ln2_g", "ln2_b", "b1", "b2")


def _align(v: int, a: int = 4096) -> int:
    return (v + a - 1) // a * a


def _pinned_view(ptr: int, nbytes: int) -> np.ndarray:
    return np.frombuffer((ctypes.c_uint8 * nbytes).from_address(ptr), dtype=np.uint8)


class HostWeights:
    """Decoder weights in host memory, filled by a provider with
    ``layer_shapes()`` (the tensors of one layer and their shapes),
    ``fill(layer, name, out)`` (fp16 tensors, layer -1 for embeddings, the
    head and the final norm) and ``fill_int4(layer, name, q, sm)``.  The
    shape's ``family`` ("opt" or "llama") says which tensors exist.

    ``pinned_matrices`` puts the layer matrices in pipo_host_alloc memory
    (streamed in place); ``pinned_head`` does the same for the output head.
    ``layout`` "fragment" stores the pinned matrices in the order the decode
    kernels read fastest (converted by the library's pipo_pack_* from the
    provider's row-major tensors); "row_major" keeps them as drawn.  Matrices
    outside pinned memory are always row-major (the library converts its
    copies).
    """

    def __init__(self, shape, wfmt: str, provider, pinned_matrices: bool = True,
                 pinned_head: bool = True, layout: str = "fragment"):
        assert wfmt in ("fp16", "int4") and layout in ("fragment", "row_major")
        self.shape, self.wfmt = shape, wfmt
        self.layout = layout if pinned_matrices else "row_major"
        d, V, L = shape.d_model, shape.vocab, shape.n_layers
        self.llama = getattr(shape, "family", "opt") == "llama"
        self._pinned: List[int] = []
        self._keep: List[object] = []
        layer_shapes = provider.layer_shapes()
        dims = {nm: layer_shapes[nm] for nm in MATRIX_SHAPES}
        small = {nm: layer_shapes[nm][0] for nm in SMALL if nm in layer_shapes}
        self.layers: List[Dict[str, object]] = []
        c_layers = (B.PipoLayerHost * L)()
        for j in range(L):
            mats: Dict[str, object] = {}
            if pinned_matrices:
                sizes = []
                for nm in MATRIX_SHAPES:
                    N, K = dims[nm]
                    if wfmt == "fp16":
                        sizes += [N * K * 2]
                    else:
                        sizes += [N * K // 2, N * (K // 64) * 4]
                total = sum(_align(s) for s in sizes)
                ptr = B.pipo_host_alloc(total)
                self._pinned.append(ptr)
                region = _pinned_view(ptr, total)
                off = 0
                views = []
                for s in sizes:
                    views.append(region[off:off + s])
                    off += _align(s)
                for i, nm in enumerate(MATRIX_SHAPES):
                    N, K = dims[nm]
                    if wfmt == "fp16":
                        mats[nm] = views[i].view(np.float16).reshape(N, K)
                    else:
                        mats[nm] = (views[2 * i].reshape(N, K // 2),
                                    views[2 * i + 1].view(np.float16).reshape(N, K // 64, 2))
            else:
                for nm in MATRIX_SHAPES:
                    N, K = dims[nm]
                    mats[nm] = (np.empty((N, K), np.float16) if wfmt == "fp16" else
                                (np.empty((N, K // 2), np.uint8),
                                 np.empty((N, K // 64, 2), np.float16)))
            for nm in MATRIX_SHAPES:
                N, K = dims[nm]
                if self.layout == "fragment":   # draw row-major, store in fragment order
                    if wfmt == "fp16":
                        B.pipo_pack_f16(provider.fill(j, nm, np.empty((N, K), np.float16)),
                                        mats[nm].reshape(-1))
                    else:
                        q = np.empty((N, K // 2), np.uint8)
                        sm = np.empty((N, K // 64, 2), np.float16)
                        provider.fill_int4(j, nm, q, sm)
                        B.pipo_pack_w4(q, sm, mats[nm][0].reshape(-1), mats[nm][1].reshape(-1))
                elif wfmt == "fp16":
                    provider.fill(j, nm, mats[nm])
                else:
                    provider.fill_int4(j, nm, mats[nm][0], mats[nm][1])
            for nm, n in small.items():
                mats[nm] = provider.fill(j, nm, np.empty(n, np.float16))
            self.layers.append(mats)
            cl = c_layers[j]
            for nm in small:
                setattr(cl, nm, mats[nm].ctypes.data)
            for nm, qn in zip(MATRIX_SHAPES, ("qqkv", "qo", "q1", "q2")):
                if wfmt == "fp16":
                    setattr(cl, nm, mats[nm].ctypes.data)
                else:
                    q4 = getattr(cl, qn)
                    q4.q = mats[nm][0].ctypes.data
                    q4.scale_min = mats[nm][1].ctypes.data
        self.c_layers = c_layers

        def table(pinned: bool) -> np.ndarray:
            if not pinned:
                return np.empty((V, d), np.float16)
            ptr = B.pipo_host_alloc(V * d * 2)
            self._pinned.append(ptr)
            return _pinned_view(ptr, V * d * 2).view(np.float16).reshape(V, d)

        # the streamed output head gets the pinned region: the token table
        # (tied) for OPT, the untied head for LLaMA
        self.tok_emb = provider.fill(-1, "tok_emb", table(pinned_head and not self.llama))
        self.lnf_g = provider.fill(-1, "lnf_g", np.empty(d, np.float16))
        if self.llama:
            self.lm_head = provider.fill(-1, "lm_head", table(pinned_head))
            self.pos_emb = self.lnf_b = None
        else:
            self.lm_head = None
            self.pos_emb = provider.fill(
                -1, "pos_emb", np.empty((shape.max_pos + shape.pos_offset, d), np.float16))
            self.lnf_b = provider.fill(-1, "lnf_b", np.empty(d, np.float16))

        def addr(a: Optional[np.ndarray]) -> Optional[int]:
            return None if a is None else a.ctypes.data

        self.c_weights = B.PipoHostWeights(addr(self.tok_emb), addr(self.pos_emb),
                                           addr(self.lnf_g), addr(self.lnf_b),
                                           ctypes.cast(c_layers, ctypes.POINTER(B.PipoLayerHost)),
                                           addr(self.lm_head),
                                           B.PIPO_LAYOUT_FRAGMENT if self.layout == "fragment"
                                           else B.PIPO_LAYOUT_ROW_MAJOR)

    def free(self):
        """Release the pinned regions (after every context using them is destroyed)."""
        self.layers = []
        self.tok_emb = self.lm_head = None
        for p in self._pinned:
            B.pipo_host_free(p)
        self._pinned = []

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def c_shape(shape) -> B.PipoShape:
    """The C shape of an OPTShape or LlamaShape."""
    c = B.PipoShape(shape.n_layers, shape.d_model, shape.n_heads, shape.d_ffn, shape.vocab,
                    shape.max_pos, shape.pos_offset, shape.ln_eps)
    if getattr(shape, "family", "opt") == "llama":
        c.family = B.PIPO_FAMILY_LLAMA
        c.n_kv_heads = shape.n_kv_heads
        c.rope_theta = shape.rope_theta
        c.rope_factor = shape.rope_factor
        c.rope_low_freq_factor = shape.rope_low_freq_factor
        c.rope_high_freq_factor = shape.rope_high_freq_factor
        c.rope_orig_max_pos = shape.rope_orig_max_pos
    return c


def c_policy(wfmt: str = "fp16", weights_on_host: bool = True, embed_on_host: bool = True,
             kv_on_host: bool = False, n_weight_slots: int = 3, n_h2d_streams: int = 0,
             chunk_bytes: int = 64 << 20, max_batch: int = 1, max_seq: int = 1,
             hbm_budget_bytes: int = 0, debug_flags: int = 0,
             copy_delay_us: int = 0, pinned_budget_bytes: int = 0,
             copy_threads: int = 0, kv_fmt: str = "fp16", weights_on_disk: bool = False,
             disk_dir: Optional[str] = None) -> B.PipoPolicy:
    assert wfmt in ("fp16", "int4") and kv_fmt in ("fp16", "int4")
    return B.PipoPolicy(B.PIPO_W_FP16 if wfmt == "fp16" else B.PIPO_W_INT4_G64,
                        int(weights_on_host), int(embed_on_host), int(kv_on_host),
                        n_weight_slots, n_h2d_streams, chunk_bytes, max_batch, max_seq,
                        hbm_budget_bytes, debug_flags, copy_delay_us, pinned_budget_bytes,
                        copy_threads,
                        B.PIPO_KV_FP16 if kv_fmt == "fp16" else B.PIPO_KV_INT4_G64,
                        int(weights_on_disk), 0,
                        disk_dir.encode() if disk_dir is not None else None)


class Decoder:
    """One pipo context over HostWeights."""

    def __init__(self, weights: HostWeights, policy: Optional[B.PipoPolicy] = None, **kw):
        """`policy` (e.g. from pipo_configure) or keyword fields for c_policy."""
        self.weights = weights
        self.vocab = weights.shape.vocab
        if policy is None:
            kw.setdefault("wfmt", weights.wfmt)
            policy = c_policy(**kw)
        self.policy = policy
        self.ctx = B.pipo_create(c_shape(weights.shape), weights.c_weights, self.policy)

    def prefill(self, tokens: np.ndarray, want_logits: bool = False
                ) -> Tuple[np.ndarray, Optional[np.ndarray]]:
        logits = (np.empty((tokens.shape[0], self.vocab), np.float32) if want_logits else None)
        return B.pipo_prefill(self.ctx, tokens, logits), logits

    def decode(self, tokens: np.ndarray, want_logits: bool = False
               ) -> Tuple[np.ndarray, Optional[np.ndarray]]:
        logits = (np.empty((tokens.shape[0], self.vocab), np.float32) if want_logits else None)
        return B.pipo_decode_step(self.ctx, tokens, logits), logits

    def generate(self, prompt: np.ndarray, gen: int, want_logits: bool = False,
                 forced: Optional[np.ndarray] = None):
        """Greedy generation of `gen` tokens per sequence.  With `forced`
        ([b][gen-1]) those tokens are fed instead of the model's own
        (teacher forcing).  Returns (tokens [b][gen], logits list or None)."""
        out, logs = [], []
        nxt, lg = self.prefill(prompt, want_logits)
        out.append(nxt)
        logs.append(lg)
        for i in range(gen - 1):
            feed = nxt if forced is None else forced[:, i]
            nxt, lg = self.decode(feed, want_logits)
            out.append(nxt)
            logs.append(lg)
        return np.stack(out, axis=1), (logs if want_logits else None)

    def stats(self) -> dict:
        return B.pipo_get_stats(self.ctx)

    def reset_stats(self) -> None:
        B.pipo_reset_stats(self.ctx)

    def set_timestamps(self, on: bool) -> None:
        B.pipo_set_timestamps(self.ctx, on)

    def close(self) -> None:
        if self.ctx:
            B.pipo_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
