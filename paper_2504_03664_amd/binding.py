"""ctypes binding of libpipo.so: the C ABI of include/pipo.h, pipo_ops.h and
pipo_sched.h under the same names.  Argument marshalling only; every step
of the decoder runs in the library's HIP kernels.

Loading fails loudly (ImportError at first use) when the library has not
been built: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# PIPO_LIB / PIPO_SCHED_LIB name another build of the same libraries (the
# host-side AddressSanitizer build of build_asan.py, for CPU tests)
LIB_PATH = os.environ.get("PIPO_LIB") or os.path.join(_PKG, "libpipo.so")
SCHED_LIB_PATH = os.environ.get("PIPO_SCHED_LIB") or os.path.join(_PKG, "libpipo_sched.so")

i32, i64, f32, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double
vp, sz = ctypes.c_void_p, ctypes.c_size_t

PIPO_OK = 0
STATUS_NAMES = {0: "PIPO_OK", -1: "PIPO_ERR_ARG", -2: "PIPO_ERR_OOM_DEVICE",
                -3: "PIPO_ERR_OOM_HOST", -4: "PIPO_ERR_HIP", -5: "PIPO_ERR_STATE",
                -6: "PIPO_ERR_UNSUPPORTED", -7: "PIPO_ERR_IO"}
PIPO_W_FP16, PIPO_W_INT4_G64 = 0, 1
PIPO_FAMILY_OPT, PIPO_FAMILY_LLAMA = 0, 1
PIPO_LAYOUT_ROW_MAJOR, PIPO_LAYOUT_FRAGMENT = 0, 1
PIPO_KV_FP16, PIPO_KV_INT4_G64 = 0, 1
PIPO_PIPE_PERFORMANCE, PIPO_PIPE_MEMORY_EFFICIENT = 0, 1
PIPO_DBG_POISON_SLOTS, PIPO_DBG_COPY_DELAY, PIPO_DBG_TIMESTAMPS = 1, 2, 4
PIPO_DBG_KV_PAGEABLE, PIPO_DBG_SEGMENT_COPIES, PIPO_DBG_UNFUSED = 8, 16, 32
PIPO_EPI_F16, PIPO_EPI_RELU_F16, PIPO_EPI_ADD_F32, PIPO_EPI_F32 = 0, 1, 2, 3
PIPO_EPI_SWIGLU = 5
PIPO_MAX_KERNEL_STATS = 16


class PipoShape(ctypes.Structure):
    _fields_ = [("n_layers", i32), ("d_model", i32), ("n_heads", i32), ("d_ffn", i32),
                ("vocab", i32), ("max_pos", i32), ("pos_offset", i32), ("ln_eps", f32),
                ("family", i32), ("n_kv_heads", i32), ("rope_theta", f32), ("rope_factor", f32),
                ("rope_low_freq_factor", f32), ("rope_high_freq_factor", f32),
                ("rope_orig_max_pos", i32)]


class PipoQ4(ctypes.Structure):
    _fields_ = [("q", vp), ("scale_min", vp)]


class PipoLayerHost(ctypes.Structure):
    _fields_ = [("ln1_g", vp), ("ln1_b", vp), ("bqkv", vp), ("bo", vp), ("ln2_g", vp),
                ("ln2_b", vp), ("b1", vp), ("b2", vp), ("wqkv", vp), ("wo", vp), ("w1", vp),
                ("w2", vp), ("qqkv", PipoQ4), ("qo", PipoQ4), ("q1", PipoQ4), ("q2", PipoQ4)]


class PipoHostWeights(ctypes.Structure):
    _fields_ = [("tok_emb", vp), ("pos_emb", vp), ("lnf_g", vp), ("lnf_b", vp),
                ("layers", ctypes.POINTER(PipoLayerHost)), ("lm_head", vp), ("layout", i32)]


class PipoPolicy(ctypes.Structure):
    _fields_ = [("wfmt", i32), ("weights_on_host", i32), ("embed_on_host", i32),
                ("kv_on_host", i32), ("n_weight_slots", i32), ("n_h2d_streams", i32),
                ("chunk_bytes", i64), ("max_batch", i32), ("max_seq", i32),
                ("hbm_budget_bytes", i64), ("debug_flags", i32), ("copy_delay_us", i32),
                ("pinned_budget_bytes", i64), ("copy_threads", i32), ("kv_fmt", i32),
                ("weights_on_disk", i32), ("reserved0", i32), ("disk_dir", ctypes.c_char_p)]


class PipoPlan(ctypes.Structure):
    _fields_ = [("weight_bytes", i64), ("kv_bytes", i64), ("hbm_bytes", i64),
                ("host_kv_bytes", i64), ("h2d_bytes_per_step", i64), ("pipeline", i32),
                ("reserved0", i32), ("host_weight_bytes", i64), ("disk_bytes", i64),
                ("disk_bytes_per_step", i64)]


class PipoResources(ctypes.Structure):
    _fields_ = [("hbm_bytes", i64), ("host_bytes", i64), ("disk_bytes", i64)]


class PipoKernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", i64), ("total_ms", f64),
                ("alg_bytes", f64), ("alg_flops", f64)]


class PipoStats(ctypes.Structure):
    _fields_ = [("h2d_bytes", i64), ("h2d_weight_bytes", i64), ("h2d_kv_bytes", i64),
                ("d2h_bytes", i64), ("n_copies", i64), ("n_kernels", i64),
                ("decode_steps", i64), ("decode_wall_ms", f64), ("prefill_wall_ms", f64),
                ("window_ms", f64), ("copy_busy_ms", f64), ("kernel_busy_ms", f64),
                ("busy_ms", f64), ("staged_bytes", i64), ("disk_read_bytes", i64),
                ("disk_read_ms", f64), ("hbm_bytes", i64),
                ("pinned_host_bytes", i64),
                ("n_kernel_stats", i32),
                ("kernels", PipoKernelStat * PIPO_MAX_KERNEL_STATS)]


class PipoSchedConfig(ctypes.Structure):
    _fields_ = [("n_layers", i32), ("n_slots", i32), ("n_h2d", i32), ("layers_streamed", i32),
                ("head_streamed", i32), ("kv_on_host", i32), ("poison", i32), ("delay", i32),
                ("chunk_bytes", i64), ("layer_seg_bytes", i64 * 10), ("head_bytes", i64),
                ("merged", i32), ("layer_seg_off", i64 * 10)]


class PipoError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        self.status = status
        super().__init__(f"{where}: {STATUS_NAMES.get(status, status)}: {msg}")


# ---------------------------------------------------------------------------
_lib = None
_sched_lib = None

_SIGNATURES = {
    "pipo_create": ([ctypes.POINTER(PipoShape), ctypes.POINTER(PipoHostWeights),
                     ctypes.POINTER(PipoPolicy), ctypes.POINTER(vp)], i32),
    "pipo_prefill": ([vp, vp, i32, i32, vp, vp], i32),
    "pipo_decode_step": ([vp, vp, vp, vp], i32),
    "pipo_get_stats": ([vp, ctypes.POINTER(PipoStats)], i32),
    "pipo_reset_stats": ([vp], i32),
    "pipo_destroy": ([vp], None),
    "pipo_set_timestamps": ([vp, i32], i32),
    "pipo_debug_fail_pass": ([vp, i64], i32),
    "pipo_plan_policy": ([ctypes.POINTER(PipoShape), ctypes.POINTER(PipoPolicy),
                          ctypes.POINTER(PipoPlan)], i32),
    "pipo_configure": ([ctypes.POINTER(PipoShape), i32, i32, i32, i32,
                        ctypes.POINTER(PipoResources), ctypes.POINTER(PipoPolicy),
                        ctypes.POINTER(PipoPlan)], i32),
    "pipo_measure_h2d_peak": ([i64, i32, i32, ctypes.POINTER(f64)], i32),
    "pipo_measure_h2d_chunked": ([i64, i64, i32, i32, ctypes.POINTER(f64)], i32),
    "pipo_measure_disk_read": ([ctypes.c_char_p, i64, i64, i32, i32, ctypes.POINTER(f64),
                                ctypes.POINTER(i32)], i32),
    "pipo_measure_disk_tier": ([vp, i64, i32, ctypes.POINTER(f64)], i32),
    "pipo_host_alloc": ([sz], vp),
    "pipo_host_free": ([vp], None),
    "pipo_last_error": ([], ctypes.c_char_p),
    "pipo_dev_alloc": ([sz, ctypes.POINTER(vp)], i32),
    "pipo_dev_free": ([vp], i32),
    "pipo_copy_h2d": ([vp, vp, sz], i32),
    "pipo_copy_d2h": ([vp, vp, sz], i32),
    "pipo_dev_synchronize": ([], i32),
    "pipo_op_gemm_f16": ([vp, vp, vp, vp, i64, i64, i64, i32, vp, i64, vp], i32),
    "pipo_op_gemm_w4": ([vp, vp, vp, vp, vp, i64, i64, i64, i32, vp, i64, vp], i32),
    "pipo_op_gemm_workspace_bytes": ([i64, i64, i64, i32], i64),
    "pipo_op_gemm_f16_frag": ([vp, vp, vp, vp, i64, i64, i64, i32, vp, i64, vp], i32),
    "pipo_op_gemm_w4_frag": ([vp, vp, vp, vp, vp, i64, i64, i64, i32, vp, i64, vp], i32),
    "pipo_pack_f16": ([vp, vp, i64, i64], i32),
    "pipo_pack_w4": ([vp, vp, vp, vp, i64, i64], i32),
    "pipo_op_layernorm": ([vp, vp, vp, vp, i64, i64, i64, i64, f32, vp], i32),
    "pipo_op_attn_decode": ([vp, vp, vp, vp, i32, i32, i32, i32, vp, i64, vp], i32),
    "pipo_op_attn_decode_workspace_bytes": ([i32, i32, i32, i32], i64),
    "pipo_op_attn_decode_noalloc": ([vp, vp, vp, vp, i32, i32, i32, i32, vp], i32),
    "pipo_op_attn_decode_kv4": ([vp, vp, vp, vp, i32, i32, i32, i32, vp, i64, vp], i32),
    "pipo_op_kv_quant": ([vp, vp, i64, i64, vp], i32),
    "pipo_op_kv_dequant": ([vp, vp, i64, i64, vp], i32),
    "pipo_op_attn_prefill": ([vp, vp, vp, vp, i32, i32, i32, i32, vp], i32),
    "pipo_op_argmax": ([vp, vp, i64, i64, vp], i32),
    "pipo_op_argmax_ws": ([vp, vp, i64, i64, vp, i64, vp], i32),
    "pipo_op_argmax_workspace_bytes": ([i64, i64], i64),
    "pipo_op_copy": ([vp, vp, i64, vp], i32),
    "pipo_op_attn_decode_gqa": ([vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, i64, vp], i32),
    "pipo_op_attn_decode_gqa_workspace_bytes": ([i32, i32, i32, i32, i32], i64),
    "pipo_op_attn_prefill_gqa": ([vp, vp, vp, vp, i32, i32, i32, i32, i32, vp], i32),
    "pipo_op_rmsnorm": ([vp, vp, vp, i64, i64, i64, i64, f32, vp], i32),
    "pipo_op_rope": ([vp, vp, vp, i64, i64, i64, i64, i64, i32, i32, i32, f32, vp], i32),
    "pipo_rope_table": ([ctypes.POINTER(PipoShape), i32, vp], i32),
    "pipo_op_swiglu": ([vp, vp, i64, i64, vp], i32),
    "pipo_op_embed": ([vp, vp, vp, vp, i64, i64, i64, i64, i64, vp], i32),
    "pipo_sched_trace": ([ctypes.POINTER(PipoSchedConfig), i32, vp, vp, vp, i64, vp, i64], i64),
}


def _declare(lib, names):
    for name in names:
        args, res = _SIGNATURES[name]
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


def lib():
    """The GPU library; raises ImportError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: run `python -m paper_2504_03664_amd.build`")
        _lib = _declare(ctypes.CDLL(LIB_PATH), _SIGNATURES.keys())
    return _lib


def sched_lib():
    """The CPU-only schedule library (no HIP runtime needed)."""
    global _sched_lib
    if _sched_lib is None:
        if not os.path.exists(SCHED_LIB_PATH):
            raise ImportError(f"{SCHED_LIB_PATH} is missing: run the build")
        _sched_lib = _declare(ctypes.CDLL(SCHED_LIB_PATH), ["pipo_sched_trace"])
    return _sched_lib


def _check(status: int, where: str):
    if status != PIPO_OK:
        raise PipoError(status, where, lib().pipo_last_error().decode())


def _ptr(a: Optional[np.ndarray]) -> Optional[int]:
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


# ---------------------------------------------------------------------------
# main ABI
def pipo_create(shape: PipoShape, weights: PipoHostWeights, policy: PipoPolicy) -> int:
    ctx = vp()
    _check(lib().pipo_create(ctypes.byref(shape), ctypes.byref(weights), ctypes.byref(policy),
                             ctypes.byref(ctx)), "pipo_create")
    return ctx.value


def pipo_prefill(ctx: int, tokens: np.ndarray, logits: Optional[np.ndarray] = None
                 ) -> np.ndarray:
    """tokens int32 [b][P]; logits: optional float32 [b][vocab] to receive the
    last position's logits.  Returns the greedy next tokens [b]."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    b, P = tokens.shape
    nxt = np.empty(b, dtype=np.int32)
    if logits is not None:
        assert logits.dtype == np.float32 and logits.shape[0] == b and logits.flags["C_CONTIGUOUS"]
    _check(lib().pipo_prefill(ctx, _ptr(tokens), b, P, _ptr(logits), _ptr(nxt)), "pipo_prefill")
    return nxt


def pipo_decode_step(ctx: int, tokens: np.ndarray, logits: Optional[np.ndarray] = None
                     ) -> np.ndarray:
    """tokens int32 [b]; returns the greedy next tokens [b]."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    b = tokens.shape[0]
    nxt = np.empty(b, dtype=np.int32)
    if logits is not None:
        assert logits.dtype == np.float32 and logits.shape[0] == b and logits.flags["C_CONTIGUOUS"]
    _check(lib().pipo_decode_step(ctx, _ptr(tokens), _ptr(logits), _ptr(nxt)), "pipo_decode_step")
    return nxt


def pipo_get_stats(ctx: int) -> dict:
    st = PipoStats()
    _check(lib().pipo_get_stats(ctx, ctypes.byref(st)), "pipo_get_stats")
    out = {name: getattr(st, name) for name, _ in PipoStats._fields_
           if name not in ("kernels", "n_kernel_stats")}
    out["kernels"] = {
        st.kernels[i].name.decode(): dict(launches=st.kernels[i].launches,
                                          total_ms=st.kernels[i].total_ms,
                                          alg_bytes=st.kernels[i].alg_bytes,
                                          alg_flops=st.kernels[i].alg_flops)
        for i in range(st.n_kernel_stats)}
    return out


def pipo_reset_stats(ctx: int) -> None:
    _check(lib().pipo_reset_stats(ctx), "pipo_reset_stats")


def _plan_dict(p: PipoPlan) -> dict:
    return {name: getattr(p, name) for name, _ in PipoPlan._fields_}


def pipo_plan_policy(shape: PipoShape, policy: PipoPolicy) -> dict:
    plan = PipoPlan()
    _check(lib().pipo_plan_policy(ctypes.byref(shape), ctypes.byref(policy), ctypes.byref(plan)),
           "pipo_plan_policy")
    return _plan_dict(plan)


def pipo_configure(shape: PipoShape, wfmt: int, kv_fmt: int, max_batch: int, max_seq: int,
                   hbm_bytes: int = 0, host_bytes: int = 0, disk_bytes: int = 0):
    """Returns (PipoPolicy, plan dict)."""
    res = PipoResources(hbm_bytes, host_bytes, disk_bytes)
    pol, plan = PipoPolicy(), PipoPlan()
    _check(lib().pipo_configure(ctypes.byref(shape), wfmt, kv_fmt, max_batch, max_seq,
                                ctypes.byref(res), ctypes.byref(pol), ctypes.byref(plan)),
           "pipo_configure")
    return pol, _plan_dict(plan)


def pipo_set_timestamps(ctx: int, on: bool) -> None:
    _check(lib().pipo_set_timestamps(ctx, int(on)), "pipo_set_timestamps")


def pipo_debug_fail_pass(ctx: int, n_ops: int) -> None:
    _check(lib().pipo_debug_fail_pass(ctx, n_ops), "pipo_debug_fail_pass")


def pipo_destroy(ctx: int) -> None:
    lib().pipo_destroy(ctx)


def pipo_measure_h2d_peak(nbytes: int, iters: int = 10, n_streams: int = 1) -> float:
    g = f64()
    _check(lib().pipo_measure_h2d_peak(nbytes, iters, n_streams, ctypes.byref(g)),
           "pipo_measure_h2d_peak")
    return g.value


def pipo_measure_h2d_chunked(nbytes: int, chunk_bytes: int, iters: int = 5,
                             n_streams: int = 1) -> float:
    g = f64()
    _check(lib().pipo_measure_h2d_chunked(nbytes, chunk_bytes, iters, n_streams, ctypes.byref(g)),
           "pipo_measure_h2d_chunked")
    return g.value


def pipo_measure_disk_read(directory: str, nbytes: int, chunk_bytes: int = 64 << 20,
                           n_threads: int = 8, iters: int = 2) -> Tuple[float, bool]:
    """(GB/s, direct I/O used) of the disk tier's read pattern in `directory`."""
    g, direct = f64(), i32()
    _check(lib().pipo_measure_disk_read(directory.encode(), nbytes, chunk_bytes, n_threads,
                                        iters, ctypes.byref(g), ctypes.byref(direct)),
           "pipo_measure_disk_read")
    return g.value, bool(direct.value)


def pipo_measure_disk_tier(ctx: int, nbytes: int, iters: int = 3) -> float:
    """GB/s of reading the context's own disk-tier file the way decode does."""
    g = f64()
    _check(lib().pipo_measure_disk_tier(ctx, nbytes, iters, ctypes.byref(g)),
           "pipo_measure_disk_tier")
    return g.value


def pipo_host_alloc(nbytes: int) -> int:
    p = lib().pipo_host_alloc(nbytes)
    if not p:
        raise MemoryError(f"pipo_host_alloc({nbytes}) failed")
    return p


def pipo_host_free(p: int) -> None:
    lib().pipo_host_free(p)


def pipo_last_error() -> str:
    return lib().pipo_last_error().decode()


# ---------------------------------------------------------------------------
# op-level ABI (device pointers as ints)
class DeviceBuffer:
    """HBM buffer owned by the caller through pipo_dev_alloc / pipo_dev_free."""

    def __init__(self, nbytes: int):
        p = vp()
        _check(lib().pipo_dev_alloc(max(int(nbytes), 1), ctypes.byref(p)), "pipo_dev_alloc")
        self.ptr, self.nbytes = p.value, int(nbytes)

    @classmethod
    def from_array(cls, a: np.ndarray) -> "DeviceBuffer":
        a = np.ascontiguousarray(a)
        buf = cls(a.nbytes)
        _check(lib().pipo_copy_h2d(buf.ptr, _ptr(a), a.nbytes), "pipo_copy_h2d")
        return buf

    def to_array(self, dtype, shape) -> np.ndarray:
        out = np.empty(shape, dtype=dtype)
        assert out.nbytes <= self.nbytes
        _check(lib().pipo_copy_d2h(_ptr(out), self.ptr, out.nbytes), "pipo_copy_d2h")
        return out

    def free(self):
        if self.ptr:
            lib().pipo_dev_free(self.ptr)
            self.ptr = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def pipo_dev_synchronize() -> None:
    _check(lib().pipo_dev_synchronize(), "pipo_dev_synchronize")


def pipo_op_gemm_f16(X, W, bias, out, M, N, K, epi, workspace=None, workspace_bytes=0,
                     stream=None):
    _check(lib().pipo_op_gemm_f16(X, W, bias, out, M, N, K, epi, workspace, workspace_bytes,
                                  stream), "pipo_op_gemm_f16")


def pipo_op_gemm_w4(X, Wq, Wsm, bias, out, M, N, K, epi, workspace=None, workspace_bytes=0,
                    stream=None):
    _check(lib().pipo_op_gemm_w4(X, Wq, Wsm, bias, out, M, N, K, epi, workspace,
                                 workspace_bytes, stream), "pipo_op_gemm_w4")


def pipo_op_gemm_f16_frag(X, W, bias, out, M, N, K, epi, workspace=None, workspace_bytes=0,
                          stream=None):
    _check(lib().pipo_op_gemm_f16_frag(X, W, bias, out, M, N, K, epi, workspace,
                                       workspace_bytes, stream), "pipo_op_gemm_f16_frag")


def pipo_op_gemm_w4_frag(X, Wq, Wsm, bias, out, M, N, K, epi, workspace=None, workspace_bytes=0,
                         stream=None):
    _check(lib().pipo_op_gemm_w4_frag(X, Wq, Wsm, bias, out, M, N, K, epi, workspace,
                                      workspace_bytes, stream), "pipo_op_gemm_w4_frag")


def pipo_pack_f16(W: np.ndarray, out: Optional[np.ndarray] = None) -> np.ndarray:
    """Row-major fp16 W [N][K] -> PIPO_LAYOUT_FRAGMENT (flat, N*K halves)."""
    W = np.ascontiguousarray(W)
    N, K = W.shape
    if out is None:
        out = np.empty(N * K, dtype=W.dtype)
    _check(lib().pipo_pack_f16(_ptr(W), _ptr(out), N, K), "pipo_pack_f16")
    return out


def pipo_pack_w4(q: np.ndarray, sm: np.ndarray, q_out: Optional[np.ndarray] = None,
                 sm_out: Optional[np.ndarray] = None):
    """Row-major INT4 (q [N][K/2], sm [N][K/64][2]) -> PIPO_LAYOUT_FRAGMENT."""
    q, sm = np.ascontiguousarray(q), np.ascontiguousarray(sm)
    N, K = q.shape[0], q.shape[1] * 2
    if q_out is None:
        q_out = np.empty(q.size, dtype=np.uint8)
    if sm_out is None:
        sm_out = np.empty(sm.size, dtype=sm.dtype)
    _check(lib().pipo_pack_w4(_ptr(q), _ptr(sm), _ptr(q_out), _ptr(sm_out), N, K),
           "pipo_pack_w4")
    return q_out, sm_out


def pipo_op_gemm_workspace_bytes(M, N, K, wfmt) -> int:
    """wfmt: PIPO_W_FP16 or PIPO_W_INT4_G64."""
    return lib().pipo_op_gemm_workspace_bytes(M, N, K, wfmt)


def pipo_op_layernorm(x, g, b, y, rows, d, src_stride, src_offset, eps, stream=None):
    _check(lib().pipo_op_layernorm(x, g, b, y, rows, d, src_stride, src_offset, eps, stream),
           "pipo_op_layernorm")


def pipo_op_attn_decode(q, kc, vc, o, b, n_heads, head_dim, t, workspace=None,
                        workspace_bytes=0, stream=None):
    _check(lib().pipo_op_attn_decode(q, kc, vc, o, b, n_heads, head_dim, t, workspace,
                                     workspace_bytes, stream), "pipo_op_attn_decode")


def pipo_op_attn_decode_noalloc(q, kc, vc, o, b, n_heads, head_dim, t, stream=None):
    _check(lib().pipo_op_attn_decode_noalloc(q, kc, vc, o, b, n_heads, head_dim, t, stream),
           "pipo_op_attn_decode_noalloc")


def pipo_op_attn_decode_workspace_bytes(b, n_heads, head_dim, t) -> int:
    return lib().pipo_op_attn_decode_workspace_bytes(b, n_heads, head_dim, t)


def pipo_op_attn_decode_kv4(q, kc, vc, o, b, n_heads, head_dim, t, workspace=None,
                            workspace_bytes=0, stream=None):
    _check(lib().pipo_op_attn_decode_kv4(q, kc, vc, o, b, n_heads, head_dim, t, workspace,
                                         workspace_bytes, stream), "pipo_op_attn_decode_kv4")


def pipo_op_kv_quant(x, out, rows, d, stream=None):
    _check(lib().pipo_op_kv_quant(x, out, rows, d, stream), "pipo_op_kv_quant")


def pipo_op_kv_dequant(src, y, rows, d, stream=None):
    _check(lib().pipo_op_kv_dequant(src, y, rows, d, stream), "pipo_op_kv_dequant")


def pipo_op_attn_prefill(q, kc, vc, o, b, P, n_heads, head_dim, stream=None):
    _check(lib().pipo_op_attn_prefill(q, kc, vc, o, b, P, n_heads, head_dim, stream),
           "pipo_op_attn_prefill")


def pipo_op_argmax(logits, nxt, rows, V, stream=None):
    _check(lib().pipo_op_argmax(logits, nxt, rows, V, stream), "pipo_op_argmax")


def pipo_op_argmax_ws(logits, nxt, rows, V, workspace=None, workspace_bytes=0, stream=None):
    _check(lib().pipo_op_argmax_ws(logits, nxt, rows, V, workspace, workspace_bytes, stream),
           "pipo_op_argmax_ws")


def pipo_op_argmax_workspace_bytes(rows, V) -> int:
    return int(lib().pipo_op_argmax_workspace_bytes(rows, V))


def pipo_op_copy(dst, src, nbytes, stream=None):
    _check(lib().pipo_op_copy(dst, src, nbytes, stream), "pipo_op_copy")


def pipo_op_attn_decode_gqa(q, kc, vc, o, b, n_heads, n_kv_heads, head_dim, t, kv_fmt,
                            workspace=None, workspace_bytes=0, stream=None):
    _check(lib().pipo_op_attn_decode_gqa(q, kc, vc, o, b, n_heads, n_kv_heads, head_dim, t,
                                         kv_fmt, workspace, workspace_bytes, stream),
           "pipo_op_attn_decode_gqa")


def pipo_op_attn_decode_gqa_workspace_bytes(b, n_heads, n_kv_heads, head_dim, t) -> int:
    return int(lib().pipo_op_attn_decode_gqa_workspace_bytes(b, n_heads, n_kv_heads, head_dim,
                                                             t))


def pipo_op_attn_prefill_gqa(q, kc, vc, o, b, P, n_heads, n_kv_heads, head_dim, stream=None):
    _check(lib().pipo_op_attn_prefill_gqa(q, kc, vc, o, b, P, n_heads, n_kv_heads, head_dim,
                                          stream), "pipo_op_attn_prefill_gqa")


def pipo_op_rmsnorm(x, g, y, rows, d, src_stride, src_offset, eps, stream=None):
    _check(lib().pipo_op_rmsnorm(x, g, y, rows, d, src_stride, src_offset, eps, stream),
           "pipo_op_rmsnorm")


def pipo_op_rope(q, k, cos_sin, M, rows_per_seq, pos0, kpos0, batch, n_heads, n_kv_heads,
                 head_dim, q_scale, stream=None):
    _check(lib().pipo_op_rope(q, k, cos_sin, M, rows_per_seq, pos0, kpos0, batch, n_heads,
                              n_kv_heads, head_dim, q_scale, stream), "pipo_op_rope")


def pipo_rope_table(shape: PipoShape, n_pos: int) -> np.ndarray:
    """[n_pos][head_dim/2][2] float32 (cos, sin) table the library uses."""
    dh = shape.d_model // shape.n_heads
    out = np.zeros((n_pos, dh // 2, 2), dtype=np.float32)
    _check(lib().pipo_rope_table(ctypes.byref(shape), n_pos, _ptr(out)), "pipo_rope_table")
    return out


def pipo_op_swiglu(gu, h, M, F, stream=None):
    _check(lib().pipo_op_swiglu(gu, h, M, F, stream), "pipo_op_swiglu")


def pipo_op_embed(ids, tok_table, pos_table, x, rows, d, rows_per_seq, pos0, pos_offset,
                  stream=None):
    _check(lib().pipo_op_embed(ids, tok_table, pos_table, x, rows, d, rows_per_seq, pos0,
                               pos_offset, stream), "pipo_op_embed")


# ---------------------------------------------------------------------------
def pipo_sched_trace(cfg: PipoSchedConfig, passes, kv_row_bytes: int = 0,
                     use_gpu_lib: bool = False) -> str:
    """passes: list of (prefill: bool, pos0, T).  Uses the CPU-only library
    unless use_gpu_lib."""
    L = lib() if use_gpu_lib else sched_lib()
    n = len(passes)
    pf = np.array([int(p[0]) for p in passes], dtype=np.int32)
    p0 = np.array([p[1] for p in passes], dtype=np.int64)
    T = np.array([p[2] for p in passes], dtype=np.int64)
    size = 1 << 20
    while True:
        buf = ctypes.create_string_buffer(size)
        r = L.pipo_sched_trace(ctypes.byref(cfg), n, _ptr(pf), _ptr(p0), _ptr(T), kv_row_bytes,
                               ctypes.addressof(buf), size)
        if r >= 0:
            return buf.value.decode()
        if size > (1 << 30):
            raise ValueError("pipo_sched_trace: invalid configuration")
        size *= 4
