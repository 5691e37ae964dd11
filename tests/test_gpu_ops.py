"""Each GPU operation through the C ABI (pipo_ops.h) against the oracle or an
exact integer reference."""
import numpy as np
import pytest

import synth
from oracle import causal_attention, dequant_int4_g64, layer_norm, quant_kv_int4_g64
from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.binding import DeviceBuffer as DB

pytestmark = pytest.mark.gpu

GEMM_SHAPES = [(1, 50, 128), (4, 100, 256), (16, 64, 128), (33, 130, 384), (64, 96, 128),
               (65, 200, 256), (128, 128, 128), (300, 257, 512),
               # big tiles (at least 512 tiles of 256 x 256), ragged M and N
               (2050, 16400, 128),
               # 64-row workgroups (N >= 12288), ragged N
               (16, 12300, 256), (40, 12288, 128), (64, 12350, 128), (7, 1000, 1024),
               # streaming kernel: K split over workgroups (up to 8 ways), INT4
               # chunk length not dividing K, ragged M and N
               (17, 130, 4096), (32, 200, 2048), (50, 1000, 1280), (100, 300, 640),
               (128, 1030, 1024), (129, 64, 256),
               # fp16 streaming grid of 129..191 eight-wave workgroups unsplit:
               # six waves per workgroup, ragged N
               (64, 18440, 128)]
EPIS = [B.PIPO_EPI_F16, B.PIPO_EPI_RELU_F16, B.PIPO_EPI_ADD_F32, B.PIPO_EPI_F32]


def log(msg):
    print(msg, flush=True)


def run_gemm(X, W, bias, epi, out_init=None, w4=None, workspace=True, frag=False):
    """One GEMM through the C ABI; `workspace` False passes none (no K split);
    `frag` packs W into fragment order (library packer) and calls the
    fragment-order entry point."""
    M, K = X.shape
    N = W.shape[0] if w4 is None else w4[0].shape[0]
    ws_bytes = B.pipo_op_gemm_workspace_bytes(M, N, K, B.PIPO_W_FP16 if w4 is None
                                              else B.PIPO_W_INT4_G64) if workspace else 0
    dWs = DB(ws_bytes) if ws_bytes > 0 else None
    ws = (dWs.ptr, ws_bytes) if dWs else (None, 0)
    dX = DB.from_array(X.astype(np.float16))
    dB = DB.from_array(bias.astype(np.float16)) if bias is not None else None
    f32 = epi in (B.PIPO_EPI_ADD_F32, B.PIPO_EPI_F32)
    if out_init is not None:
        dO = DB.from_array(out_init.astype(np.float32))
    else:
        dO = DB(M * N * (4 if f32 else 2))
    if w4 is None:
        W16 = W.astype(np.float16)
        dW = DB.from_array(B.pipo_pack_f16(W16) if frag else W16)
        op = B.pipo_op_gemm_f16_frag if frag else B.pipo_op_gemm_f16
        op(dX.ptr, dW.ptr, dB.ptr if dB else None, dO.ptr, M, N, K, epi, *ws)
    else:
        q, sm = B.pipo_pack_w4(*w4) if frag else w4
        dq, dsm = DB.from_array(q), DB.from_array(sm)
        op = B.pipo_op_gemm_w4_frag if frag else B.pipo_op_gemm_w4
        op(dX.ptr, dq.ptr, dsm.ptr, dB.ptr if dB else None, dO.ptr, M, N, K, epi, *ws)
    B.pipo_dev_synchronize()
    return dO.to_array(np.float32 if f32 else np.float16, (M, N))


def expected(acc, bias, epi, out_init):
    v = acc + (bias if bias is not None else 0)
    if epi == B.PIPO_EPI_RELU_F16:
        v = np.maximum(v, 0)
    if epi == B.PIPO_EPI_ADD_F32:
        v = out_init + v
    if epi in (B.PIPO_EPI_F16, B.PIPO_EPI_RELU_F16):
        v = v.astype(np.float16).astype(np.float64)   # the exact fp32 sum, rounded once
    return v


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
@pytest.mark.parametrize("epi", EPIS)
def test_gemm_f16_exact_on_integers(M, N, K, epi):
    log(f"gemm_f16 exact M={M} N={N} K={K} epi={epi}")
    if K > 2048:     # keep |sum| <= 2048 so that fp16 outputs stay exact
        K = 2048
    rng = np.random.default_rng(M * 7 + N + K + epi)
    X = rng.integers(-2, 3, (M, K)).astype(np.float64)
    W = rng.integers(-2, 3, (N, K)).astype(np.float64)
    bias = rng.integers(-8, 9, N).astype(np.float64)
    init = rng.integers(-100, 100, (M, N)).astype(np.float64) if epi == B.PIPO_EPI_ADD_F32 else None
    got = run_gemm(X, W, bias, epi, init)
    want = expected(X @ W.T, bias, epi, init)
    assert np.array_equal(got.astype(np.float64), want)


@pytest.mark.parametrize("M,N,K", GEMM_SHAPES)
def test_gemm_w4_exact_on_integers(M, N, K):
    log(f"gemm_w4 exact M={M} N={N} K={K}")
    rng = np.random.default_rng(M + 3 * N + K)
    codes = rng.integers(0, 16, (N, K))
    q = (codes[:, 0::2] | (codes[:, 1::2] << 4)).astype(np.uint8)
    sm = np.empty((N, K // 64, 2), np.float16)
    sm[..., 0] = rng.choice([0.25, 0.5, 1.0], (N, K // 64))
    sm[..., 1] = rng.choice([-2.0, -1.0, 0.0], (N, K // 64))
    X = rng.integers(-1, 2, (M, K)).astype(np.float64)
    Wd = dequant_int4_g64(q, sm, np.float64)
    for epi in (B.PIPO_EPI_F32, B.PIPO_EPI_RELU_F16):
        got = run_gemm(X, None, None, epi, w4=(q, sm))
        assert np.array_equal(got.astype(np.float64), expected(X @ Wd.T, None, epi, None))


@pytest.mark.parametrize("M,N,K", [(3, 384, 1024), (64, 384, 1024), (200, 384, 1024),
                                   (2050, 16400, 128)])
def test_gemm_random_vs_oracle_definition(M, N, K):
    log(f"gemm random M={M} N={N} K={K}")
    rng = np.random.default_rng(M)
    X = (rng.standard_normal((M, K)) * 0.5).astype(np.float16)
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float16)
    bias = (rng.standard_normal(N) * 0.02).astype(np.float16)
    want = X.astype(np.float64) @ W.astype(np.float64).T + bias.astype(np.float64)
    for frag in (False, True):
        got = run_gemm(X, W, bias, B.PIPO_EPI_F32, frag=frag)
        assert np.abs(got - want).max() <= 1e-4 * np.abs(want).max() + 1e-5
    q, sm = synth.quant_int4_g64(W)
    got4 = run_gemm(X, None, bias, B.PIPO_EPI_F32, w4=(q, sm))
    want4 = X.astype(np.float64) @ dequant_int4_g64(q, sm, np.float64).T + bias.astype(np.float64)
    # the kernel rounds each expanded weight to fp16 (relative 2^-11)
    assert np.abs(got4 - want4).max() <= 2e-3 * np.abs(want4).max()


@pytest.mark.parametrize("M,N,K", [(1, 64, 128), (16, 12288, 256), (7, 1008, 1024),
                                   (33, 144, 384), (64, 1024, 4096), (128, 1040, 1024),
                                   (129, 64, 256), (300, 272, 512),
                                   # big tiles (at least 512 of 256 x 256): ragged M
                                   # and N, and exact multiples
                                   (2050, 16400, 128), (4100, 8208, 256),
                                   (2048, 16384, 384)])
@pytest.mark.parametrize("w4", [False, True])
def test_gemm_fragment_order_equals_row_major(M, N, K, w4):
    """W in fragment order (skinny, streaming with K splits, tiled and
    big-tile kernels): the same products in the same order, bit for bit.
    With fp16 W at big-tile shapes the two sides are different kernels
    (global -> LDS loads against the 128 x 128 tiles)."""
    log(f"gemm fragment order M={M} N={N} K={K} w4={w4}")
    rng = np.random.default_rng(M + N + K + w4)
    X = rng.standard_normal((M, K)).astype(np.float16)
    W = (rng.standard_normal((N, K)) * 0.05).astype(np.float16)
    bias = (rng.standard_normal(N) * 0.05).astype(np.float16)
    q = synth.quant_int4_g64(W) if w4 else None
    for epi in (B.PIPO_EPI_F32, B.PIPO_EPI_RELU_F16):
        a = run_gemm(X, W, bias, epi, w4=q)
        b = run_gemm(X, W, bias, epi, w4=q, frag=True)
        assert np.array_equal(a.view(np.uint16 if a.dtype == np.float16 else np.uint32),
                              b.view(np.uint16 if b.dtype == np.float16 else np.uint32))


@pytest.mark.parametrize("w4", [False, True])
@pytest.mark.parametrize("frag", [False, True])
def test_gemm_big_tiles_equal_tiled(w4, frag):
    """At M = 2050, N = 16400 (585 tiles of 256 x 256) the big-tile kernels
    run; the first 300 rows alone (130 tiles) run on the 128 x 128 kernel.
    Both sum every output over the same k blocks in the same order: the
    same bits."""
    log(f"gemm big vs tiled w4={w4} frag={frag}")
    rng = np.random.default_rng(11 + w4 + 2 * frag)
    M, N, K = 2050, 16400, 256
    X = rng.standard_normal((M, K)).astype(np.float16)
    W = (rng.standard_normal((N, K)) * 0.05).astype(np.float16)
    bias = (rng.standard_normal(N) * 0.05).astype(np.float16)
    q = synth.quant_int4_g64(W) if w4 else None
    for epi in (B.PIPO_EPI_F32, B.PIPO_EPI_F16):
        big = run_gemm(X, W, bias, epi, w4=q, frag=frag)
        small = run_gemm(X[:300], W, bias, epi, w4=q, frag=frag)
        view = np.uint32 if epi == B.PIPO_EPI_F32 else np.uint16
        assert np.array_equal(big[:300].view(view), small.view(view))


@pytest.mark.parametrize("M", [4, 40, 100, 200])
@pytest.mark.parametrize("w4", [False, True])
def test_gemm_deterministic_and_split_consistent(M, w4):
    """Repeated calls give the same bits; the K-split result equals the
    unsplit one up to fp32 rounding; without a split (M <= 16, M > 128, or
    no workspace) a launch over a row range of W gives those rows bit for
    bit (the summation order then depends on M and K only)."""
    log(f"gemm determinism/split M={M} w4={w4}")
    rng = np.random.default_rng(5)
    K, N = 2048, 1024
    X = (rng.standard_normal((M, K))).astype(np.float16)
    W = (rng.standard_normal((N, K)) * 0.05).astype(np.float16)
    q = synth.quant_int4_g64(W) if w4 else None
    a = run_gemm(X, W, None, B.PIPO_EPI_F32, w4=q)
    b = run_gemm(X, W, None, B.PIPO_EPI_F32, w4=q)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    unsplit = run_gemm(X, W, None, B.PIPO_EPI_F32, w4=q, workspace=False)
    assert np.abs(a - unsplit).max() <= 1e-5 * np.abs(unsplit).max()
    for n0, n1 in ((0, 32), (32, 160), (160, 1000)):
        part = W[n0:n1]
        got = run_gemm(X, part, None, B.PIPO_EPI_F32,
                       w4=synth.quant_int4_g64(part) if w4 else None, workspace=False)
        assert np.array_equal(got.view(np.uint32), unsplit[:, n0:n1].view(np.uint32))


@pytest.mark.parametrize("w4", [False, True])
def test_gemm_split_merge_workspace_alignment(w4):
    """The K-split merge reads four partial columns at a time from a 16-byte
    aligned workspace and one at a time otherwise: a workspace 4 bytes off
    that alignment gives the same bits."""
    log(f"gemm split merge alignment w4={w4}")
    rng = np.random.default_rng(11)
    M, N, K = 40, 1024, 2048
    X = rng.standard_normal((M, K)).astype(np.float16)
    W = (rng.standard_normal((N, K)) * 0.05).astype(np.float16)
    wfmt = B.PIPO_W_INT4_G64 if w4 else B.PIPO_W_FP16
    ws_bytes = B.pipo_op_gemm_workspace_bytes(M, N, K, wfmt)
    assert ws_bytes > 0
    dX, dO = DB.from_array(X), DB(M * N * 4)
    dWs = DB(ws_bytes + 256)
    if w4:
        q, sm = synth.quant_int4_g64(W)
        dq, dsm = DB.from_array(q), DB.from_array(sm)
        call = lambda ws: B.pipo_op_gemm_w4(dX.ptr, dq.ptr, dsm.ptr, None, dO.ptr, M, N, K,
                                            B.PIPO_EPI_F32, ws, ws_bytes)
    else:
        dW = DB.from_array(W)
        call = lambda ws: B.pipo_op_gemm_f16(dX.ptr, dW.ptr, None, dO.ptr, M, N, K,
                                             B.PIPO_EPI_F32, ws, ws_bytes)
    outs = []
    for off in (0, 4):
        call(dWs.ptr + off)
        B.pipo_dev_synchronize()
        outs.append(dO.to_array(np.float32, (M, N)))
    assert np.array_equal(outs[0].view(np.uint32), outs[1].view(np.uint32))


def test_attention_workspace_reuse():
    """Repeated split calls on one workspace give identical results."""
    log("attention workspace reuse")
    rng = np.random.default_rng(9)
    b, H, D, t = 4, 4, 128, 999
    q, kc, vc = _attn_inputs(rng, b, t + 1, H, D)
    na = B.pipo_op_attn_decode_workspace_bytes(b, H, D, t)
    assert na > 0
    wa = DB(na)
    dq, dk, dv, do = DB.from_array(q), DB.from_array(kc), DB.from_array(vc), DB(b * H * D * 2)
    outs = []
    for _ in range(3):
        B.pipo_op_attn_decode(dq.ptr, dk.ptr, dv.ptr, do.ptr, b, H, D, t, wa.ptr, na)
        B.pipo_dev_synchronize()
        outs.append(do.to_array(np.uint16, (b, H * D)))
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


@pytest.mark.parametrize("rows,d,stride,offset", [(1, 768, 1, 0), (5, 4096, 1, 0),
                                                  (3, 7168, 4, 3), (33, 128, 2, 0)])
def test_layernorm_vs_oracle(rows, d, stride, offset):
    log(f"layernorm rows={rows} d={d}")
    rng = np.random.default_rng(d + rows)
    x = (rng.standard_normal((rows * stride, d)) * 3 + 1).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float16)
    b = (0.1 * rng.standard_normal(d)).astype(np.float16)
    dx, dg, db = DB.from_array(x), DB.from_array(g), DB.from_array(b)
    dy = DB(rows * d * 2)
    B.pipo_op_layernorm(dx.ptr, dg.ptr, db.ptr, dy.ptr, rows, d, stride, offset, 1e-5)
    B.pipo_dev_synchronize()
    got = dy.to_array(np.float16, (rows, d)).astype(np.float64)
    src = x.astype(np.float64)[offset::stride][:rows]
    want = layer_norm(src, g.astype(np.float64), b.astype(np.float64), 1e-5)
    assert np.abs(got - want).max() <= 4e-3 * np.abs(want).max()


def _attn_inputs(rng, b, T, H, D):
    d = H * D
    q = (rng.standard_normal((b, d)) * 0.3).astype(np.float16)
    kc = rng.standard_normal((T, b, d)).astype(np.float16)
    vc = rng.standard_normal((T, b, d)).astype(np.float16)
    return q, kc, vc


@pytest.mark.parametrize("b,T,H,D", [(1, 1, 2, 64), (3, 7, 4, 128), (2, 64, 2, 64),
                                     (2, 65, 3, 128), (1, 544, 2, 128), (4, 300, 1, 64),
                                     (2, 2000, 2, 128), (16, 543, 4, 128),
                                     # one head per workgroup with key splits
                                     (3, 600, 56, 128), (5, 129, 6, 64), (2, 700, 5, 128),
                                     # 4 and 2 heads per workgroup (b * H >= 6144, 3072),
                                     # unsplit
                                     (112, 40, 56, 128), (56, 41, 56, 128), (60, 33, 52, 64),
                                     # the longest context the kernel takes
                                     (1, 65536, 2, 128)])
@pytest.mark.parametrize("split", [False, True])
def test_attn_decode_vs_oracle(b, T, H, D, split):
    log(f"attn_decode b={b} T={T} H={H} D={D} split={split}")
    rng = np.random.default_rng(T * 10 + b)
    q, kc, vc = _attn_inputs(rng, b, T, H, D)
    dq, dk, dv = DB.from_array(q), DB.from_array(kc), DB.from_array(vc)
    do = DB(b * H * D * 2)
    ws_bytes = B.pipo_op_attn_decode_workspace_bytes(b, H, D, T - 1) if split else 0
    ws = DB(ws_bytes) if ws_bytes else None
    B.pipo_op_attn_decode(dq.ptr, dk.ptr, dv.ptr, do.ptr, b, H, D, T - 1,
                          ws.ptr if ws else None, ws_bytes)
    B.pipo_dev_synchronize()
    got = do.to_array(np.float16, (b, H * D)).astype(np.float64)
    for i in range(b):
        want = causal_attention(q[i:i + 1].astype(np.float64), kc[:, i].astype(np.float64),
                                vc[:, i].astype(np.float64), H)[0]
        assert np.abs(got[i] - want).max() <= 5e-3 * max(1.0, np.abs(want).max())


def _kv_rows(codes, sm):
    """INT4 cache rows as the library stores them: each row's d/2 code bytes,
    then its d/64 fp16 (scale, min) pairs."""
    R = codes.shape[0]
    return np.ascontiguousarray(np.concatenate([codes, sm.view(np.uint8).reshape(R, -1)], axis=1))


def _kv_test_rows(rng, R, d):
    scales = np.array([1e-3, 0.02, 1.0, 300.0])[rng.integers(0, 4, R)]
    x = (rng.standard_normal((R, d)) * scales[:, None]).astype(np.float16)
    if R > 3:
        x[1, 64:128] = np.float16(-2.5)                     # constant group: scale 0
        half = np.arange(64) % 15 + 0.5                     # min 0, max 15: scale 1, the
        half[:2] = 0, 15                                    # rest half-way between codes
        x[2, :64] = half.astype(np.float16)
        x[3, :64] = (np.arange(64) % 16) * 0.125 - 1.0      # exact grid points
    return x


@pytest.mark.parametrize("rows,d", [(1, 256), (37, 512), (300, 768), (5, 7168)])
def test_kv_quant_dequant_bit_exact_vs_oracle(rows, d):
    """The GPU quantizer makes the oracle's codes, scales and mins bit for
    bit (the same fp32 decisions); the expansion is code * scale + min
    rounded once to fp16."""
    log(f"kv quant rows={rows} d={d}")
    rng = np.random.default_rng(rows + d)
    x = _kv_test_rows(rng, rows, d)
    codes, sm = quant_kv_int4_g64(x)
    want = _kv_rows(codes, sm)
    dx, dq = DB.from_array(x), DB(want.nbytes)
    B.pipo_op_kv_quant(dx.ptr, dq.ptr, rows, d)
    B.pipo_dev_synchronize()
    got = dq.to_array(np.uint8, want.shape)
    assert np.array_equal(got, want)
    dy = DB(rows * d * 2)
    B.pipo_op_kv_dequant(dq.ptr, dy.ptr, rows, d)
    B.pipo_dev_synchronize()
    back = dy.to_array(np.float16, (rows, d))
    assert np.array_equal(back, dequant_int4_g64(codes, sm, np.float64).astype(np.float16))


@pytest.mark.parametrize("b,T,H,D", [(1, 1, 4, 64), (3, 70, 4, 128), (2, 1000, 2, 128),
                                     (16, 543, 8, 64), (4, 600, 56, 128), (3, 129, 6, 128),
                                     (2, 300, 12, 64)])
@pytest.mark.parametrize("split", [False, True])
def test_attn_decode_kv4(b, T, H, D, split):
    """Decode attention over an INT4 cache (32 elements per lane, its own
    summation order) matches the fp16 kernel over the expanded cache to
    fp32 rounding, and the oracle over the dequantized cache."""
    log(f"attn_decode_kv4 b={b} T={T} H={H} D={D} split={split}")
    rng = np.random.default_rng(T + 7 * b)
    d = H * D
    q, kc, vc = _attn_inputs(rng, b, T, H, D)
    ck, sk = quant_kv_int4_g64(kc.reshape(T * b, d))
    cv, sv = quant_kv_int4_g64(vc.reshape(T * b, d))
    k16 = dequant_int4_g64(ck, sk, np.float64).astype(np.float16).reshape(T, b, d)
    v16 = dequant_int4_g64(cv, sv, np.float64).astype(np.float16).reshape(T, b, d)
    dq, dk4, dv4 = DB.from_array(q), DB.from_array(_kv_rows(ck, sk)), DB.from_array(_kv_rows(cv, sv))
    dk, dv = DB.from_array(k16), DB.from_array(v16)
    ws_bytes = B.pipo_op_attn_decode_workspace_bytes(b, H, D, T - 1) if split else 0
    ws = DB(ws_bytes) if ws_bytes else None
    w = (ws.ptr if ws else None, ws_bytes)
    o4, o16 = DB(b * d * 2), DB(b * d * 2)
    B.pipo_op_attn_decode_kv4(dq.ptr, dk4.ptr, dv4.ptr, o4.ptr, b, H, D, T - 1, *w)
    B.pipo_op_attn_decode(dq.ptr, dk.ptr, dv.ptr, o16.ptr, b, H, D, T - 1, *w)
    B.pipo_dev_synchronize()
    got = o4.to_array(np.float16, (b, d)).astype(np.float64)
    ref16 = o16.to_array(np.float16, (b, d)).astype(np.float64)
    assert np.abs(got - ref16).max() <= 2e-3 * max(1.0, np.abs(ref16).max())
    for i in range(b):
        want = causal_attention(q[i:i + 1].astype(np.float64), k16[:, i].astype(np.float64),
                                v16[:, i].astype(np.float64), H)[0]
        assert np.abs(got[i] - want).max() <= 5e-3 * max(1.0, np.abs(want).max())


@pytest.mark.parametrize("b,P,H,D", [(1, 1, 2, 64), (2, 5, 2, 128), (1, 64, 3, 64),
                                     (2, 100, 2, 128), (1, 130, 1, 64), (3, 33, 4, 128),
                                     # several 128-query blocks and 64-key blocks, ragged
                                     (2, 300, 2, 128), (1, 513, 3, 64), (1, 256, 2, 128),
                                     # a long prompt: 16 query blocks, 32 key blocks
                                     (1, 2048, 2, 128)])
def test_attn_prefill_vs_oracle(b, P, H, D):
    log(f"attn_prefill b={b} P={P} H={H} D={D}")
    rng = np.random.default_rng(P * 3 + b)
    d = H * D
    q = (rng.standard_normal((b, P, d)) * 0.3).astype(np.float16)
    kc = rng.standard_normal((P, b, d)).astype(np.float16)
    vc = rng.standard_normal((P, b, d)).astype(np.float16)
    dq, dk, dv = DB.from_array(q), DB.from_array(kc), DB.from_array(vc)
    do = DB(b * P * d * 2)
    B.pipo_op_attn_prefill(dq.ptr, dk.ptr, dv.ptr, do.ptr, b, P, H, D)
    B.pipo_dev_synchronize()
    got = do.to_array(np.float16, (b, P, d)).astype(np.float64)
    for i in range(b):
        want = causal_attention(q[i].astype(np.float64), kc[:, i].astype(np.float64),
                                vc[:, i].astype(np.float64), H)
        # P is rounded to fp16 before P.V (relative 2^-11 per weight)
        assert np.abs(got[i] - want).max() <= 8e-3 * max(1.0, np.abs(want).max())


@pytest.mark.parametrize("V", [50272, 128256, 4096, 4099, 7])
def test_argmax_ties_and_ragged(V):
    """Single-pass and split (partitions merged by a second kernel) argmax:
    the largest logit, ties to the lowest index, NaNs skipped, a row of
    -inf gives its first index, a row of NaNs gives 0."""
    log(f"argmax V={V}")
    rng = np.random.default_rng(V)
    R = 8
    L = rng.standard_normal((R, V)).astype(np.float32)
    L[1, min(17, V - 1)] = L[1, V - 1] = L[1].max() + 1   # tie: lowest index wins
    L[2, :] = -np.inf
    L[2, min(5, V - 1):] = 0.0                             # first finite maximum
    L[3, V - 1] = 100.0                                    # ragged tail
    L[4, :] = 7.0                                          # all equal -> 0
    L[5, ::3] = np.nan                                     # NaNs are skipped
    L[6, :] = -np.inf                                      # all -inf -> 0
    L[7, :] = np.nan                                       # all NaN -> 0
    want = [int(np.nanargmax(r)) if not np.isnan(r).all() else 0 for r in L]
    dl = DB.from_array(L)
    ws_bytes = B.pipo_op_argmax_workspace_bytes(R, V)
    assert (ws_bytes > 0) == (V > 4096)
    ws = DB(ws_bytes) if ws_bytes else None
    for split in (False, True):
        dn = DB(R * 4)
        if split:
            B.pipo_op_argmax_ws(dl.ptr, dn.ptr, R, V, ws.ptr if ws else None, ws_bytes)
        else:
            B.pipo_op_argmax(dl.ptr, dn.ptr, R, V)
        B.pipo_dev_synchronize()
        got = dn.to_array(np.int32, (R,))
        assert got.tolist() == want, (split, got.tolist(), want)
