"""Seeded synthetic inputs for OPT-shaped decoder workloads.

This package draws and encodes inputs only: random fp16 weights, their
group-wise int4 codes, and prompt token ids.  It holds none of the decoder's
arithmetic.  The CPU oracle (``oracle/``) and the GPU library both consume
what it produces; neither of them is imported here.

Every tensor has its own counter-based stream (Philox4x64-10, see
``csrc/synth.c``), keyed by ``(seed, tensor_key(layer, name))``, so a tensor,
or a row range of it, can be regenerated independently of all others.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "synth.c")
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

WEIGHT_STD = 0.02
DEFAULT_SEED = 20250404


def build(force: bool = True) -> str:
    """Compile ``libsynth.so`` next to this file with gcc (OpenMP, F16C)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O3", "-fPIC", "-shared", "-fopenmp", "-mf16c", "-mavx2", "-mfma", "-fno-math-errno", "-std=c11",
               "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        L = ctypes.CDLL(_LIB_PATH)
        u64, i64, i32 = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int
        vp = ctypes.c_void_p
        L.synth_philox4x64_10.argtypes = [vp, vp, vp]
        L.synth_f32_to_f16.argtypes = [ctypes.c_float]
        L.synth_f32_to_f16.restype = ctypes.c_uint16
        L.synth_normal_f16.argtypes = [u64, u64, u64, u64, ctypes.c_double, vp, i32]
        L.synth_fill_f16.argtypes = [ctypes.c_uint16, u64, vp]
        L.synth_quant_int4_g64.argtypes = [vp, i64, i64, vp, vp, i32]
        L.synth_normal_int4_g64.argtypes = [u64, u64, i64, i64, ctypes.c_double, vp, vp, i32]
        _lib = L
    return _lib


def n_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.isdigit():
        n = min(n, int(env)) if int(env) > 0 else n
    return max(1, n)


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def philox4x64_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().synth_philox4x64_10(_ptr(c), _ptr(k), _ptr(out))
    return out


# ----------------------------------------------------------------------------
# tensor naming
_TENSOR_CODES = {
    "tok_emb": 1, "pos_emb": 2, "lnf_g": 3, "lnf_b": 4, "lm_head": 5,
    "ln1_g": 10, "ln1_b": 11, "wqkv": 12, "bqkv": 13, "wo": 14, "bo": 15,
    "ln2_g": 16, "ln2_b": 17, "w1": 18, "b1": 19, "w2": 20, "b2": 21,
}
MATRICES = ("wqkv", "wo", "w1", "w2")
SMALL = ("ln1_g", "ln1_b", "bqkv", "bo", "ln2_g", "ln2_b", "b1", "b2")


def tensor_key(layer: int, name: str) -> int:
    """Stream id of a tensor: layer -1 for the embeddings and the final LN."""
    return ((layer + 1) << 16) | _TENSOR_CODES[name]


def normal_f16(seed: int, key: int, n: int, std: float = WEIGHT_STD, first: int = 0,
               out: Optional[np.ndarray] = None) -> np.ndarray:
    """fp16 values std*z[first:first+n] of stream (seed, key)."""
    if out is None:
        out = np.empty(n, dtype=np.float16)
    flat = out.reshape(-1)
    assert flat.size == n and flat.dtype.itemsize == 2
    lib().synth_normal_f16(seed, key, first, n, std, _ptr(flat), n_threads())
    return out


def f32_to_f16_bits(x: float) -> int:
    return int(lib().synth_f32_to_f16(float(x)))


def quant_int4_g64(w16: np.ndarray):
    """Encode fp16 W[N][K] as (q[N][K/2] uint8, sm[N][K/64][2] fp16)."""
    w16 = np.ascontiguousarray(w16, dtype=np.float16)
    N, K = w16.shape
    assert K % 64 == 0
    q = np.empty((N, K // 2), dtype=np.uint8)
    sm = np.empty((N, K // 64, 2), dtype=np.float16)
    lib().synth_quant_int4_g64(_ptr(w16), N, K, _ptr(q), _ptr(sm), n_threads())
    return q, sm


def normal_int4_g64(seed: int, key: int, N: int, K: int, std: float = WEIGHT_STD,
                    q: Optional[np.ndarray] = None, sm: Optional[np.ndarray] = None):
    """int4 codes of normal_f16(seed, key, N*K) viewed as [N][K], without the fp16 copy."""
    assert K % 64 == 0
    if q is None:
        q = np.empty((N, K // 2), dtype=np.uint8)
    if sm is None:
        sm = np.empty((N, K // 64, 2), dtype=np.float16)
    assert q.size == N * K // 2 and sm.size == N * K // 32
    lib().synth_normal_int4_g64(seed, key, N, K, std, _ptr(q.reshape(-1)),
                                _ptr(sm.reshape(-1)), n_threads())
    return q, sm


# ----------------------------------------------------------------------------
# model shapes and workloads
@dataclasses.dataclass(frozen=True)
class OPTShape:
    n_layers: int
    d_model: int
    n_heads: int
    d_ffn: int
    vocab: int = 50272
    max_pos: int = 2048
    pos_offset: int = 2
    ln_eps: float = 1e-5

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def with_layers(self, n: int) -> "OPTShape":
        return dataclasses.replace(self, n_layers=n)


OPTShape.family = "opt"

OPT_125M = OPTShape(12, 768, 12, 3072)
OPT_6_7B = OPTShape(32, 4096, 32, 16384)
OPT_13B = OPTShape(40, 5120, 40, 20480)
OPT_30B = OPTShape(48, 7168, 56, 28672)


@dataclasses.dataclass(frozen=True)
class LlamaShape:
    """LLaMA-3.1-style decoder: RMSNorm, grouped-query attention with rotary
    positions (with the 3.1 frequency scaling), SwiGLU MLP, untied head."""
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    d_ffn: int
    vocab: int = 128256
    max_pos: int = 8192
    rope_theta: float = 500000.0
    rope_factor: float = 8.0        # 0: no frequency scaling
    rope_low_freq_factor: float = 1.0
    rope_high_freq_factor: float = 4.0
    rope_orig_max_pos: int = 8192
    ln_eps: float = 1e-5
    family = "llama"
    pos_offset = 0

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads

    def with_layers(self, n: int) -> "LlamaShape":
        return dataclasses.replace(self, n_layers=n)


LLAMA31_8B = LlamaShape(32, 4096, 32, 8, 14336)
LLAMA31_70B = LlamaShape(80, 8192, 64, 8, 28672)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    shape: object         # OPTShape or LlamaShape
    batch: int
    prompt: int
    gen: int
    wfmt: str            # "fp16" or "int4"
    kv_on_host: bool
    kv_fmt: str = "fp16"  # KV cache rows: "fp16" or "int4"
    weights_on_disk: bool = False  # layers streamed from the disk tier's file


WORKLOADS = (
    Workload("opt-125m b4 p32 g8 fp16", OPT_125M, 4, 32, 8, "fp16", False),
    Workload("opt-6.7b b16 p512 g32 fp16", OPT_6_7B, 16, 512, 32, "fp16", False),
    Workload("opt-13b b32 p512 g32 int4-g64", OPT_13B, 32, 512, 32, "int4", False),
    Workload("opt-30b b64 p512 g32 fp16", OPT_30B, 64, 512, 32, "fp16", False),
    Workload("opt-30b b128 p512 g32 int4-g64 kv-host", OPT_30B, 128, 512, 32, "int4", True),
    # the previous workload with the KV cache in INT4 as well
    Workload("opt-30b b128 p512 g32 int4-g64 kv-host kv-int4", OPT_30B, 128, 512, 32, "int4", True,
             "int4"),
    # the paper's other dense family (Section 4.1): LLaMA3.1-8B shape
    Workload("llama3.1-8b b16 p512 g32 fp16", LLAMA31_8B, 16, 512, 32, "fp16", False),
    Workload("llama3.1-8b b32 p512 g32 int4-g64", LLAMA31_8B, 32, 512, 32, "int4", False),
    # the OPT-30B decode with the layers on disk (Section 3.1.1's third tier)
    Workload("opt-30b b64 p512 g32 fp16 disk", OPT_30B, 64, 512, 32, "fp16", False,
             weights_on_disk=True),
)


def prompt_tokens(batch: int, prompt: int, vocab: int, seed: int = 1,
                  stream: int = 0) -> np.ndarray:
    """Uniform token ids in [0, vocab), int32 [batch][prompt]."""
    rng = np.random.Generator(np.random.Philox(key=np.array([seed, 0x70726F6D + stream],
                                                            dtype=np.uint64)))
    return rng.integers(0, vocab, size=(batch, prompt), dtype=np.int64).astype(np.int32)


class SyntheticOPT:
    """Random-init OPT-shaped weights, drawn per tensor on demand.

    fp16 tensors are returned as float16 arrays.  With ``wfmt == "int4"`` the
    four per-layer matrices come as ``{name: (q, sm)}`` int4 codes of the same
    fp16 draw; embeddings, LayerNorm parameters and biases stay fp16.
    LayerNorm gamma is 1 (or 1 + N(0, gain_std), rounded to fp16, so that
    tests can tell the norms apart) and beta 0; biases are N(0, std) unless
    ``zero_bias``.
    """

    def __init__(self, shape: OPTShape, seed: int = DEFAULT_SEED, wfmt: str = "fp16",
                 zero_bias: bool = False, std: float = WEIGHT_STD, gain_std: float = 0.0):
        assert wfmt in ("fp16", "int4")
        self.shape, self.seed, self.wfmt = shape, seed, wfmt
        self.zero_bias, self.std, self.gain_std = zero_bias, std, gain_std

    # shapes of every tensor of one layer
    def layer_shapes(self) -> Dict[str, tuple]:
        d, F = self.shape.d_model, self.shape.d_ffn
        return {"ln1_g": (d,), "ln1_b": (d,), "wqkv": (3 * d, d), "bqkv": (3 * d,),
                "wo": (d, d), "bo": (d,), "ln2_g": (d,), "ln2_b": (d,),
                "w1": (F, d), "b1": (F,), "w2": (d, F), "b2": (d,)}

    def fill(self, layer: int, name: str, out: np.ndarray) -> np.ndarray:
        """Write fp16 tensor (layer, name) into ``out``."""
        if name.endswith("_g"):
            if self.gain_std > 0:
                z = normal_f16(self.seed, tensor_key(layer, name), out.size, self.gain_std)
                out[...] = (z.astype(np.float32) + 1).reshape(out.shape).astype(np.float16)
            else:
                out[...] = np.float16(1.0)
        elif name.endswith("_b") and name.startswith("ln"):
            out[...] = np.float16(0.0)
        elif name.startswith("b") and self.zero_bias:
            out[...] = np.float16(0.0)
        else:
            normal_f16(self.seed, tensor_key(layer, name), out.size, self.std, out=out)
        return out

    def fill_int4(self, layer: int, name: str, q: np.ndarray, sm: np.ndarray):
        N, K = self.layer_shapes()[name]
        return normal_int4_g64(self.seed, tensor_key(layer, name), N, K, self.std, q, sm)

    def tensor(self, layer: int, name: str) -> np.ndarray:
        shp = (self.layer_shapes()[name] if layer >= 0 else
               {"tok_emb": (self.shape.vocab, self.shape.d_model),
                "pos_emb": (self.shape.max_pos + self.shape.pos_offset, self.shape.d_model),
                "lnf_g": (self.shape.d_model,), "lnf_b": (self.shape.d_model,)}[name])
        return self.fill(layer, name, np.empty(shp, dtype=np.float16))

    def tok_emb(self) -> np.ndarray:
        return self.tensor(-1, "tok_emb")

    def pos_emb(self) -> np.ndarray:
        return self.tensor(-1, "pos_emb")

    def lnf(self):
        return self.tensor(-1, "lnf_g"), self.tensor(-1, "lnf_b")

    def layer(self, j: int) -> Dict[str, object]:
        out: Dict[str, object] = {}
        for name, shp in self.layer_shapes().items():
            if name in MATRICES and self.wfmt == "int4":
                N, K = shp
                q = np.empty((N, K // 2), dtype=np.uint8)
                sm = np.empty((N, K // 64, 2), dtype=np.float16)
                out[name] = self.fill_int4(j, name, q, sm)
            else:
                out[name] = self.tensor(j, name)
        return out


class SyntheticLlama(SyntheticOPT):
    """Random-init LLaMA-3.1-shaped weights (same streams and encodings as
    SyntheticOPT): RMSNorm weights 1, no biases, q/k/v stacked in ``wqkv``
    ([(h + 2 h_kv) head_dim][d]), gate and up stacked in ``w1`` ([2 d_ffn][d],
    gate rows first), untied ``lm_head``; no position table."""

    def __init__(self, shape: "LlamaShape", seed: int = DEFAULT_SEED, wfmt: str = "fp16",
                 std: float = WEIGHT_STD, gain_std: float = 0.0):
        super().__init__(shape, seed=seed, wfmt=wfmt, zero_bias=True, std=std, gain_std=gain_std)

    def layer_shapes(self) -> Dict[str, tuple]:
        s = self.shape
        d, F, dh = s.d_model, s.d_ffn, s.head_dim
        return {"ln1_g": (d,), "wqkv": ((s.n_heads + 2 * s.n_kv_heads) * dh, d), "wo": (d, d),
                "ln2_g": (d,), "w1": (2 * F, d), "w2": (d, F)}

    def tensor(self, layer: int, name: str) -> np.ndarray:
        if layer < 0 and name in ("tok_emb", "lm_head"):
            shp = (self.shape.vocab, self.shape.d_model)
            return self.fill(layer, name, np.empty(shp, dtype=np.float16))
        if layer < 0 and name == "lnf_g":
            return self.fill(layer, name, np.empty(self.shape.d_model, dtype=np.float16))
        return super().tensor(layer, name)

    def lm_head(self) -> np.ndarray:
        return self.tensor(-1, "lm_head")

    def pos_emb(self):
        return None

    def lnf(self):
        return self.tensor(-1, "lnf_g"), None


def synthetic_model(shape, seed: int = DEFAULT_SEED, wfmt: str = "fp16", **kw):
    """The random-init weight provider of the shape's family."""
    if getattr(shape, "family", "opt") == "llama":
        return SyntheticLlama(shape, seed=seed, wfmt=wfmt, **kw)
    return SyntheticOPT(shape, seed=seed, wfmt=wfmt, **kw)


def teacher_tokens(wl: Workload, stream: int, batch: Optional[int] = None):
    """The inputs of a teacher-forced run of workload ``wl``: the prompt
    ids [b][prompt] and the ids fed at the gen - 1 decode steps [b][gen - 1]
    (both uniform in [0, vocab), seeded, independent streams), so a run's
    inputs never depend on what either implementation generated."""
    b = wl.batch if batch is None else batch
    prompt = prompt_tokens(b, wl.prompt, wl.shape.vocab, seed=1, stream=stream)
    forced = prompt_tokens(b, wl.gen - 1, wl.shape.vocab, seed=2, stream=stream)
    return prompt, forced


class ZeroKV:
    """A weight provider whose key and value projections are zero: every key
    and value row is its bias (an fp16 value).  Wraps another provider; the
    query rows, every other tensor and the encodings are the base's."""

    def __init__(self, base):
        self.base, self.shape, self.wfmt = base, base.shape, base.wfmt

    def _kv_rows(self) -> slice:
        return slice(self.shape.d_model, None)

    def fill(self, layer, name, out):
        self.base.fill(layer, name, out)
        if name == "wqkv":
            out[self._kv_rows()] = 0
        return out

    def fill_int4(self, layer, name, q, sm):
        # an INT4 row of zeros: codes 0, scale 0, min 0
        self.base.fill_int4(layer, name, q, sm)
        if name == "wqkv":
            q[self._kv_rows()] = 0
            sm[self._kv_rows()] = 0
        return q, sm

    def layer(self, j):
        L = dict(self.base.layer(j))
        w = L["wqkv"]
        if isinstance(w, tuple):
            q, sm = np.array(w[0]), np.array(w[1])
            q[self._kv_rows()] = 0
            sm[self._kv_rows()] = 0
            L["wqkv"] = (q, sm)
        else:
            w = np.array(w)
            w[self._kv_rows()] = 0
            L["wqkv"] = w
        return L

    def layer_shapes(self):
        return self.base.layer_shapes()

    def tensor(self, layer, name):
        return self.base.tensor(layer, name)

    def tok_emb(self):
        return self.base.tok_emb()

    def pos_emb(self):
        return self.base.pos_emb()

    def lnf(self):
        return self.base.lnf()
