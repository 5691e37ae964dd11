"""The LLaMA-family GPU operations through the C ABI (pipo_ops.h) against
the oracle: RMSNorm, rotary positions, SwiGLU, grouped-query attention
(decode over fp16 and INT4 caches, prefill), embedding without positions."""
import numpy as np
import pytest

import synth
from oracle import (apply_rope, dequant_int4_g64, gqa_attention, quant_kv_int4_g64, rms_norm,
                    rope_frequencies, swiglu)
from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.binding import DeviceBuffer as DB

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("rows,d,stride,offset", [(1, 4096, 1, 0), (7, 8192, 1, 0),
                                                  (3, 512, 4, 3), (33, 128, 2, 1)])
def test_rmsnorm_vs_oracle(rows, d, stride, offset):
    log(f"rmsnorm rows={rows} d={d}")
    rng = np.random.default_rng(d + rows)
    x = (rng.standard_normal((rows * stride, d)) * 3 + 0.5).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float16)
    dx, dg, dy = DB.from_array(x), DB.from_array(g), DB(rows * d * 2)
    B.pipo_op_rmsnorm(dx.ptr, dg.ptr, dy.ptr, rows, d, stride, offset, 1e-5)
    B.pipo_dev_synchronize()
    got = dy.to_array(np.float16, (rows, d)).astype(np.float64)
    want = rms_norm(x.astype(np.float64)[offset::stride][:rows], g.astype(np.float64), 1e-5)
    # fp32 statistics, one fp16 rounding of the output
    assert np.abs(got - want).max() <= 2e-3 * np.abs(want).max()


def _table(dh, n_pos, theta=500000.0, factor=8.0):
    """The oracle's (cos, sin) of p * w_i, stored as fp32 for the kernel."""
    w = rope_frequencies(dh, theta, factor, 1.0, 4.0, 8192)
    ang = np.arange(n_pos, dtype=np.float64)[:, None] * w[None, :]
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32), w


@pytest.mark.parametrize("b,T,pos0,H,Hkv,D,staging", [
    (1, 1, 0, 8, 2, 64, False), (4, 1, 511, 32, 8, 128, False), (3, 37, 0, 8, 2, 128, False),
    (2, 70, 5, 4, 4, 64, True), (5, 1, 1000, 64, 8, 128, True)])
def test_rope_vs_oracle(b, T, pos0, H, Hkv, D, staging):
    """q rows [b*T][H*D] rotated and scaled; the new keys rotated where the
    QKV epilogue wrote them: cache rows (pos0 + p) * b + i, or staging rows
    p * b + i (kpos0 = 0)."""
    log(f"rope b={b} T={T} pos0={pos0} H={H}/{Hkv} D={D} staging={staging}")
    rng = np.random.default_rng(T * 7 + pos0 + D)
    n_pos = pos0 + T
    cs, w = _table(D, n_pos)
    M = b * T
    q = rng.standard_normal((M, H * D)).astype(np.float16)
    kpos0 = 0 if staging else pos0
    rows_k = (kpos0 + T) * b
    k = rng.standard_normal((rows_k, Hkv * D)).astype(np.float16)
    dq, dk, dcs = DB.from_array(q), DB.from_array(k), DB.from_array(cs)
    scale = D ** -0.5
    B.pipo_op_rope(dq.ptr, dk.ptr, dcs.ptr, M, T, pos0, kpos0, b, H, Hkv, D, scale)
    B.pipo_dev_synchronize()
    gq = dq.to_array(np.float16, (M, H * D)).astype(np.float64)
    gk = dk.to_array(np.float16, (rows_k, Hkv * D)).astype(np.float64)
    for i in range(b):
        pos = pos0 + np.arange(T)
        want_q = apply_rope(q[i * T:(i + 1) * T].astype(np.float64) * scale, pos, w)
        assert np.abs(gq[i * T:(i + 1) * T] - want_q).max() <= 2e-3 * np.abs(want_q).max()
        krows = (kpos0 + np.arange(T)) * b + i
        want_k = apply_rope(k[krows].astype(np.float64), pos, w)
        assert np.abs(gk[krows] - want_k).max() <= 2e-3 * np.abs(want_k).max()
    # rows the rotation must not touch: earlier cache positions
    untouched = np.ones(rows_k, bool)
    untouched[(kpos0 + np.arange(T))[:, None] * b + np.arange(b)[None, :]] = False
    assert np.array_equal(gk[untouched], k[untouched].astype(np.float64))


@pytest.mark.parametrize("M,F", [(1, 14336), (16, 1024), (37, 28672), (300, 128)])
def test_swiglu_vs_oracle(M, F):
    log(f"swiglu M={M} F={F}")
    rng = np.random.default_rng(M + F)
    gu = (rng.standard_normal((M, 2 * F)) * 4).astype(np.float16)
    gu[0, :8] = [0, -20, 20, -80, 80, 1, -1, 0.5]     # saturating and small gates
    dgu, dh = DB.from_array(gu), DB(M * F * 2)
    B.pipo_op_swiglu(dgu.ptr, dh.ptr, M, F)
    B.pipo_dev_synchronize()
    got = dh.to_array(np.float16, (M, F)).astype(np.float64)
    g64 = gu.astype(np.float64)
    want = swiglu(g64[:, :F], g64[:, F:])
    assert np.all(np.abs(got - want) <= 2e-3 * np.abs(want) + 1e-6)


@pytest.mark.parametrize("M,F,K", [(1, 14336, 4096), (16, 1000, 256), (7, 64, 512),
                                   (3, 40, 128)])
@pytest.mark.parametrize("w4", [False, True])
@pytest.mark.parametrize("frag", [False, True])
def test_gemm_swiglu_epilogue(M, F, K, w4, frag):
    """The SwiGLU epilogue of the decode GEMM (gate rows over up rows, M <=
    16) gives the bits of the GEMM's fp16 output followed by the SwiGLU
    kernel, and the oracle's SwiGLU of the exact products within fp16
    rounding."""
    if frag and (2 * F) % 16:
        pytest.skip("fragment order needs N % 16 == 0")
    log(f"gemm swiglu M={M} F={F} K={K} w4={w4} frag={frag}")
    rng = np.random.default_rng(M + F + K + 2 * w4 + frag)
    X = (rng.standard_normal((M, K)) * 0.5).astype(np.float16)
    W = (rng.standard_normal((2 * F, K)) * 0.05).astype(np.float16)
    dX = DB.from_array(X)
    dgu, dh, dh2 = DB(M * 2 * F * 2), DB(M * F * 2), DB(M * F * 2)
    if w4:
        q, sm = synth.quant_int4_g64(W)
        Wd = dequant_int4_g64(q, sm, np.float64)
        if frag:
            q, sm = B.pipo_pack_w4(q, sm)
        dq, dsm = DB.from_array(q), DB.from_array(sm)
        op = B.pipo_op_gemm_w4_frag if frag else B.pipo_op_gemm_w4
        call = lambda epi, out: op(dX.ptr, dq.ptr, dsm.ptr, None, out.ptr, M, 2 * F, K, epi, None, 0)
    else:
        Wd = W.astype(np.float64)
        dW = DB.from_array(B.pipo_pack_f16(W) if frag else W)
        op = B.pipo_op_gemm_f16_frag if frag else B.pipo_op_gemm_f16
        call = lambda epi, out: op(dX.ptr, dW.ptr, None, out.ptr, M, 2 * F, K, epi, None, 0)
    call(B.PIPO_EPI_F16, dgu)
    B.pipo_op_swiglu(dgu.ptr, dh2.ptr, M, F)
    call(B.PIPO_EPI_SWIGLU, dh)
    B.pipo_dev_synchronize()
    fused = dh.to_array(np.uint16, (M, F))
    assert np.array_equal(fused, dh2.to_array(np.uint16, (M, F)))
    acc = X.astype(np.float64) @ Wd.T
    want = swiglu(acc[:, :F], acc[:, F:])
    got = fused.view(np.float16).astype(np.float64)
    assert np.all(np.abs(got - want) <= 4e-3 * np.abs(want) + 2e-3 * np.abs(want).max())


def test_gemm_swiglu_epilogue_limits():
    """The SwiGLU epilogue runs only where the decode GEMM does (M <= 16) and
    needs N = 2F even; other calls fail cleanly."""
    rng = np.random.default_rng(3)
    K, F = 128, 64
    for M, N, status in ((17, 2 * F, -6), (4, 2 * F + 1, -1)):   # UNSUPPORTED, ARG
        dX = DB.from_array((rng.standard_normal((M, K))).astype(np.float16))
        dW = DB.from_array((rng.standard_normal((N, K))).astype(np.float16))
        dh = DB(M * N * 2)
        with pytest.raises(B.PipoError) as e:
            B.pipo_op_gemm_f16(dX.ptr, dW.ptr, None, dh.ptr, M, N, K, B.PIPO_EPI_SWIGLU, None, 0)
        assert e.value.status == status


def _kv_rows(codes, sm):
    R = codes.shape[0]
    return np.ascontiguousarray(np.concatenate([codes, sm.view(np.uint8).reshape(R, -1)], axis=1))


_GQA_SHAPES = [(1, 1, 8, 2, 64), (3, 70, 8, 4, 128), (16, 543, 32, 8, 128),
               (2, 2000, 64, 8, 128), (4, 300, 16, 2, 64), (2, 65, 4, 2, 128)]
# INT4 rows need a multiple of 256 elements (the library rejects others), so
# only those shapes are generated with kv_fmt "int4".
_GQA_CASES = [(*s, fmt) for s in _GQA_SHAPES for fmt in ("fp16", "int4")
              if fmt == "fp16" or (s[3] * s[4]) % 256 == 0]


@pytest.mark.parametrize("b,T,H,Hkv,D,kv_fmt", _GQA_CASES)
@pytest.mark.parametrize("split", [False, True])
def test_attn_decode_gqa_vs_oracle(b, T, H, Hkv, D, kv_fmt, split):
    """One workgroup per key/value head serves its G query heads: against
    the oracle's grouped-query attention (over the dequantized cache for
    INT4 rows, which the kernel must read bit for bit like the fp16 path)."""
    dkv = Hkv * D
    log(f"attn_decode_gqa b={b} T={T} H={H}/{Hkv} D={D} {kv_fmt} split={split}")
    rng = np.random.default_rng(T * 13 + b + H)
    q = (rng.standard_normal((b, H * D)) * 0.3).astype(np.float16)
    kc = rng.standard_normal((T, b, dkv)).astype(np.float16)
    vc = rng.standard_normal((T, b, dkv)).astype(np.float16)
    fmt = B.PIPO_KV_FP16
    if kv_fmt == "int4":
        ck, sk = quant_kv_int4_g64(kc.reshape(T * b, dkv))
        cv, sv = quant_kv_int4_g64(vc.reshape(T * b, dkv))
        kc = dequant_int4_g64(ck, sk, np.float64).astype(np.float16).reshape(T, b, dkv)
        vc = dequant_int4_g64(cv, sv, np.float64).astype(np.float16).reshape(T, b, dkv)
        dk, dv = DB.from_array(_kv_rows(ck, sk)), DB.from_array(_kv_rows(cv, sv))
        fmt = B.PIPO_KV_INT4_G64
    else:
        dk, dv = DB.from_array(kc), DB.from_array(vc)
    dq, do = DB.from_array(q), DB(b * H * D * 2)
    ws_bytes = B.pipo_op_attn_decode_gqa_workspace_bytes(b, H, Hkv, D, T - 1) if split else 0
    ws = DB(ws_bytes) if ws_bytes else None
    B.pipo_op_attn_decode_gqa(dq.ptr, dk.ptr, dv.ptr, do.ptr, b, H, Hkv, D, T - 1, fmt,
                              ws.ptr if ws else None, ws_bytes)
    B.pipo_dev_synchronize()
    got = do.to_array(np.float16, (b, H * D)).astype(np.float64)
    for i in range(b):
        want = gqa_attention(q[i:i + 1].astype(np.float64), kc[:, i].astype(np.float64),
                             vc[:, i].astype(np.float64), H, Hkv)[0]
        assert np.abs(got[i] - want).max() <= 5e-3 * max(1.0, np.abs(want).max())
    if kv_fmt == "int4":   # the INT4 read equals the fp16 kernel over the expanded rows
        dk16, dv16, do16 = DB.from_array(kc), DB.from_array(vc), DB(b * H * D * 2)
        B.pipo_op_attn_decode_gqa(dq.ptr, dk16.ptr, dv16.ptr, do16.ptr, b, H, Hkv, D, T - 1,
                                  B.PIPO_KV_FP16, ws.ptr if ws else None, ws_bytes)
        B.pipo_dev_synchronize()
        assert np.array_equal(do.to_array(np.uint16, (b, H * D)),
                              do16.to_array(np.uint16, (b, H * D)))


def test_attn_decode_gqa_with_one_group_is_the_mha_kernel():
    """n_kv_heads == n_heads takes the multi-head path bit for bit."""
    rng = np.random.default_rng(5)
    b, T, H, D = 4, 300, 8, 128
    q = (rng.standard_normal((b, H * D)) * 0.3).astype(np.float16)
    kc = rng.standard_normal((T, b, H * D)).astype(np.float16)
    vc = rng.standard_normal((T, b, H * D)).astype(np.float16)
    dq, dk, dv = DB.from_array(q), DB.from_array(kc), DB.from_array(vc)
    o1, o2 = DB(b * H * D * 2), DB(b * H * D * 2)
    ws_bytes = B.pipo_op_attn_decode_workspace_bytes(b, H, D, T - 1)
    ws = DB(ws_bytes) if ws_bytes else None
    w = (ws.ptr if ws else None, ws_bytes)
    B.pipo_op_attn_decode(dq.ptr, dk.ptr, dv.ptr, o1.ptr, b, H, D, T - 1, *w)
    B.pipo_op_attn_decode_gqa(dq.ptr, dk.ptr, dv.ptr, o2.ptr, b, H, H, D, T - 1, B.PIPO_KV_FP16,
                              *w)
    B.pipo_dev_synchronize()
    assert np.array_equal(o1.to_array(np.uint16, (b, H * D)), o2.to_array(np.uint16, (b, H * D)))


@pytest.mark.parametrize("b,P,H,Hkv,D", [(1, 1, 4, 2, 64), (2, 37, 8, 2, 128),
                                         (1, 130, 8, 1, 64), (2, 64, 32, 8, 128),
                                         (1, 300, 8, 2, 128)])
def test_attn_prefill_gqa_vs_oracle(b, P, H, Hkv, D):
    log(f"attn_prefill_gqa b={b} P={P} H={H}/{Hkv} D={D}")
    rng = np.random.default_rng(P * 5 + b + H)
    dkv = Hkv * D
    q = (rng.standard_normal((b, P, H * D)) * 0.3).astype(np.float16)
    kc = rng.standard_normal((P, b, dkv)).astype(np.float16)
    vc = rng.standard_normal((P, b, dkv)).astype(np.float16)
    dq, dk, dv = DB.from_array(q), DB.from_array(kc), DB.from_array(vc)
    do = DB(b * P * H * D * 2)
    B.pipo_op_attn_prefill_gqa(dq.ptr, dk.ptr, dv.ptr, do.ptr, b, P, H, Hkv, D)
    B.pipo_dev_synchronize()
    got = do.to_array(np.float16, (b, P, H * D)).astype(np.float64)
    for i in range(b):
        want = gqa_attention(q[i].astype(np.float64), kc[:, i].astype(np.float64),
                             vc[:, i].astype(np.float64), H, Hkv)
        # P is rounded to fp16 before P.V (relative 2^-11 per weight)
        assert np.abs(got[i] - want).max() <= 8e-3 * max(1.0, np.abs(want).max())


def test_embed_without_position_table():
    rng = np.random.default_rng(3)
    V, d, rows = 300, 512, 37
    tok = rng.standard_normal((V, d)).astype(np.float16)
    ids = rng.integers(0, V, rows).astype(np.int32)
    dt, di, dx = DB.from_array(tok), DB.from_array(ids), DB(rows * d * 4)
    B.pipo_op_embed(di.ptr, dt.ptr, None, dx.ptr, rows, d, rows, 0, 0)
    B.pipo_dev_synchronize()
    assert np.array_equal(dx.to_array(np.float32, (rows, d)), tok[ids].astype(np.float32))
