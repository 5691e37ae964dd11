"""The C ABI without a GPU: every declared symbol is exported, and invalid
shapes and policies are rejected before any device work."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.model import c_policy, c_shape

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("pipo.h", "pipo_ops.h", "pipo_sched.h")]


def declared_functions():
    names = []
    for h in HEADERS:
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names += re.findall(r"\b(pipo_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def exported(path):
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    return {line.split()[-1] for line in out.splitlines() if line.strip()}


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 20
    syms = exported(B.LIB_PATH)
    missing = [n for n in names if n not in syms]
    assert not missing, missing
    L = B.lib()
    for n in names:
        assert getattr(L, n) is not None


def test_schedule_library_exports_trace():
    assert "pipo_sched_trace" in exported(B.SCHED_LIB_PATH)


class _Shape:
    def __init__(self, **kw):
        base = dict(n_layers=2, d_model=256, n_heads=2, d_ffn=512, vocab=100, max_pos=64,
                    pos_offset=2, ln_eps=1e-5)
        base.update(kw)
        self.__dict__.update(base)


def _create(shape, **pol):
    dummy = np.zeros(8, np.uint16)
    layers = (B.PipoLayerHost * max(shape.n_layers, 1))()
    w = B.PipoHostWeights(dummy.ctypes.data, dummy.ctypes.data, dummy.ctypes.data,
                          dummy.ctypes.data, ctypes.cast(layers, ctypes.POINTER(B.PipoLayerHost)))
    pol.setdefault("max_batch", 1)
    pol.setdefault("max_seq", 8)
    return B.pipo_create(c_shape(shape), w, c_policy(**pol))


@pytest.mark.parametrize("kw,status", [
    (dict(n_layers=0), "PIPO_ERR_ARG"),
    (dict(n_heads=3), "PIPO_ERR_ARG"),                 # d_model not a multiple of n_heads
    (dict(n_heads=8), "PIPO_ERR_UNSUPPORTED"),         # head_dim 32
    (dict(d_model=320, n_heads=5), "PIPO_ERR_UNSUPPORTED"),  # d not a multiple of 128
    (dict(d_ffn=500), "PIPO_ERR_UNSUPPORTED"),
    (dict(vocab=0), "PIPO_ERR_ARG"),
])
def test_bad_shapes_rejected(kw, status):
    with pytest.raises(B.PipoError) as e:
        _create(_Shape(**kw))
    assert B.STATUS_NAMES[e.value.status] == status
    assert B.pipo_last_error() != ""


@pytest.mark.parametrize("pol,status", [
    (dict(max_batch=0), "PIPO_ERR_ARG"),
    (dict(max_seq=65), "PIPO_ERR_UNSUPPORTED"),        # beyond max_pos
    (dict(n_weight_slots=17), "PIPO_ERR_ARG"),
    (dict(n_h2d_streams=3), "PIPO_ERR_ARG"),
    (dict(kv_on_host=True, weights_on_host=False), "PIPO_ERR_UNSUPPORTED"),
])
def test_bad_policies_rejected(pol, status):
    with pytest.raises(B.PipoError) as e:
        _create(_Shape(), **pol)
    assert B.STATUS_NAMES[e.value.status] == status


def test_null_weights_rejected():
    with pytest.raises(B.PipoError) as e:
        B.pipo_create(c_shape(_Shape()), B.PipoHostWeights(), c_policy(max_batch=1, max_seq=4))
    assert e.value.status == -1


def test_gemm_workspace_sizes():
    """GEMM K splits (host-side planning only, no GPU needed) happen only for
    16 < M <= 128 and stay within the cap of 8."""
    for M in (1, 16, 129, 4096):
        assert B.pipo_op_gemm_workspace_bytes(M, 100, 4096, B.PIPO_W_FP16) == 0
    for wfmt in (B.PIPO_W_FP16, B.PIPO_W_INT4_G64):
        for M, N, K in ((17, 130, 4096), (64, 7168, 7168), (128, 28672, 7168), (32, 5120, 20480)):
            ws = B.pipo_op_gemm_workspace_bytes(M, N, K, wfmt)
            assert ws % (M * N * 4) == 0 and ws // (M * N * 4) in (0, 2, 4, 8)
        assert B.pipo_op_gemm_workspace_bytes(17, 130, 4096, wfmt) == 8 * 17 * 130 * 4


def test_disk_probe_runs_without_a_gpu(tmp_path):
    """The disk tier's read pattern (direct I/O through a pageable chunk,
    several threads) on a small file; the probe removes its file."""
    gbps, direct = B.pipo_measure_disk_read(str(tmp_path), 8 << 20, 1 << 20, 3, 1)
    assert gbps > 0
    assert list(tmp_path.iterdir()) == []
    with pytest.raises(B.PipoError) as e:
        B.pipo_measure_disk_read(str(tmp_path / "missing"), 1 << 20)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_IO"
    with pytest.raises(B.PipoError) as e:
        B.pipo_measure_disk_read(str(tmp_path), 1 << 20, n_threads=0)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_ARG"


def _frag_f16_reference(W):
    """Fragment order as pipo.h defines it: block (rg, kb) of 16 rows x 32 k,
    inside which slot r + 16 g holds row r, k = 8 g .. 8 g + 7."""
    N, K = W.shape
    out = np.empty(N * K, W.dtype)
    for rg in range(N // 16):
        for kb in range(K // 32):
            base = (rg * (K // 32) + kb) * 512
            for r in range(16):
                for g in range(4):
                    out[base + (r + 16 * g) * 8:base + (r + 16 * g) * 8 + 8] = \
                        W[16 * rg + r, 32 * kb + 8 * g:32 * kb + 8 * g + 8]
    return out


def test_pack_f16_matches_the_layout_definition():
    rng = np.random.default_rng(0)
    for N, K in ((16, 32), (48, 128), (32, 256)):
        W = rng.integers(0, 1 << 16, size=(N, K)).astype(np.uint16)
        got = B.pipo_pack_f16(W)
        assert np.array_equal(got, _frag_f16_reference(W))
        assert sorted(got.tolist()) == sorted(W.reshape(-1).tolist())   # a permutation


def test_pack_w4_matches_the_layout_definition():
    rng = np.random.default_rng(1)
    N, K = 32, 256
    q = rng.integers(0, 256, size=(N, K // 2)).astype(np.uint8)
    sm = rng.integers(0, 1 << 16, size=(N, K // 64, 2)).astype(np.uint16)
    gq, gsm = B.pipo_pack_w4(q, sm)
    for n in range(N):
        for k in range(0, K, 2):   # codes (k, k+1) share a byte
            byte = (n // 16 * (K // 128) + k // 128) * 1024 + \
                (n % 16 + 16 * ((k % 128) // 32)) * 16 + (k % 32) // 2
            assert gq[byte] == q[n, k // 2]
        for grp in range(K // 64):
            pair = (n // 16 * (K // 128) + grp // 2) * 32 + (n % 16) * 2 + grp % 2
            assert gsm[2 * pair] == sm[n, grp, 0] and gsm[2 * pair + 1] == sm[n, grp, 1]
    with pytest.raises(B.PipoError):
        B.pipo_pack_w4(q[:, :40], sm[:, :1])   # K = 80 is not a multiple of 128


def test_attention_workspace_and_limits_without_a_gpu():
    """Decode-attention workspace sizing and the prefill size limit are host
    logic: splits only while a grid would have fewer than 768 workgroups, the
    workspace covers the fp16 and the INT4 cache, and a prefill whose 64-row
    key block would span 2^31 elements is refused before any launch."""
    # batch 16, 56 heads: fp16 rows take one head per workgroup (896 of
    # them, no split), INT4 rows four (224, so 4 splits): sized for the latter
    assert B.pipo_op_attn_decode_workspace_bytes(16, 56, 128, 543) == 16 * 56 * 4 * 130 * 4
    # batch 64: 1792 two-head (fp16) or 896 four-head (INT4) workgroups, no split
    assert B.pipo_op_attn_decode_workspace_bytes(64, 56, 128, 543) == 0
    assert B.pipo_op_attn_decode_gqa_workspace_bytes(64, 56, 56, 128, 543) == 0
    # batch 1: keys split, S * (head_dim + 2) floats per head, S <= 16
    ws = B.pipo_op_attn_decode_workspace_bytes(1, 56, 128, 16383)
    assert 0 < ws <= 56 * 16 * 130 * 4 and ws % (56 * 130 * 4) == 0
    # batch 128, 56 heads: 1792 four-head workgroups for either cache, no split
    assert B.pipo_op_attn_decode_workspace_bytes(128, 56, 128, 543) == 0
    with pytest.raises(B.PipoError) as e:                 # never dereferenced
        B.pipo_op_attn_prefill(8, 8, 8, 8, 40000, 1, 56, 128)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_UNSUPPORTED"


def test_decode_attention_context_limit_without_a_gpu():
    """t + 1 keys beyond 65536 are refused before any launch (the largest
    context is run on the GPU in test_gpu_ops.py)."""
    for fn in (lambda t: B.pipo_op_attn_decode(8, 8, 8, 8, 1, 2, 128, t),
               lambda t: B.pipo_op_attn_decode_gqa(8, 8, 8, 8, 1, 8, 2, 128, t, B.PIPO_KV_FP16)):
        with pytest.raises(B.PipoError) as e:
            fn(65536)
        assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_UNSUPPORTED"


def test_bench_kernel_symbols_follow_the_library_plan():
    """bench.py names the kernels a projection launches (to find their
    counters in the committed profiles) by restating the library's K-split
    rule; the split it implies must be the one the library plans, for every
    projection of every decode workload (the library's workspace query gives
    S · M · N · 4 bytes for S > 1 splits)."""
    import sys
    sys.path.insert(0, ROOT)
    import bench
    import synth
    for wl in synth.WORKLOADS:
        sh = wl.shape
        d, M = sh.d_model, wl.batch
        llama = getattr(sh, "family", "opt") == "llama"
        hkv = sh.n_kv_heads if llama else sh.n_heads
        dh = d // sh.n_heads
        F = sh.d_ffn
        mats = {"qkv": (d + 2 * hkv * dh, d), "oproj": (d, d),
                "fc1": (2 * F if llama else F, d), "fc2": (d, F)}
        w4 = wl.wfmt == "int4"
        for name, (N, K) in mats.items():
            epi = {"qkv": 4, "oproj": 2, "fc2": 2,
                   "fc1": (5 if M <= 16 else 0) if llama else 1}[name]
            syms = bench.gemm_symbols(M, N, K, epi, w4, True)
            ws = B.pipo_op_gemm_workspace_bytes(M, N, K, B.PIPO_W_INT4_G64 if w4 else B.PIPO_W_FP16)
            splits = ws // (M * N * 4)
            combine = [s for s in syms if s.startswith("gemm_combine<")]
            if splits > 1:
                assert combine and combine[0].startswith(f"gemm_combine<{epi}, {splits}, "), \
                    (wl.name, name, syms, splits)
            else:
                assert not combine, (wl.name, name, syms)


def test_bench_profile_tags_are_distinct():
    """bench.py keys the committed traffic summaries by model, batch, KV
    placement and KV format: every workload with its own kernels has its own
    key (the disk-tier run shares the kernels, and the key, of the workload
    it streams), and every committed summary belongs to a workload."""
    import sys
    sys.path.insert(0, ROOT)
    import bench
    import synth
    keys = {}
    for wl in synth.WORKLOADS:
        kernels = " ".join(t for t in wl.name.split() if t != "disk")
        assert keys.setdefault(bench.profile_tag(wl.name), kernels) == kernels, wl.name
    assert len(keys) == len({" ".join(t for t in w.name.split() if t != "disk")
                             for w in synth.WORKLOADS})
    for f in os.listdir(os.path.join(ROOT, "profiles")):
        if f.startswith("hbm_traffic_") and f.endswith(".json"):
            assert f[len("hbm_traffic_"):-len(".json")] in keys, f
