"""Decode attention through the entry point that allocates nothing
(pipo_op_attn_decode_noalloc) against the same operation with a caller
workspace (pipo_op_attn_decode): the same kernels and split choice, so the
same bits; and against the oracle's attention.  Two calls in a row, the
second with a smaller input, so the fixed array is reused with the first
call's partials still in it."""
import numpy as np
import pytest

from oracle import causal_attention
from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.binding import DeviceBuffer as DB

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


def _inputs(seed, b, T, H, D):
    rng = np.random.default_rng(seed)
    d = H * D
    q = (rng.standard_normal((b, d)) * 0.3).astype(np.float16)
    kc = rng.standard_normal((T, b, d)).astype(np.float16)
    vc = rng.standard_normal((T, b, d)).astype(np.float16)
    return q, kc, vc


def _both(b, T, H, D, seed):
    q, kc, vc = _inputs(seed, b, T, H, D)
    dq, dk, dv = DB.from_array(q), DB.from_array(kc), DB.from_array(vc)
    o_ws, o_na = DB(b * H * D * 2), DB(b * H * D * 2)
    ws_bytes = B.pipo_op_attn_decode_workspace_bytes(b, H, D, T - 1)
    ws = DB(ws_bytes) if ws_bytes else None
    B.pipo_op_attn_decode(dq.ptr, dk.ptr, dv.ptr, o_ws.ptr, b, H, D, T - 1,
                          ws.ptr if ws else None, ws_bytes)
    B.pipo_op_attn_decode_noalloc(dq.ptr, dk.ptr, dv.ptr, o_na.ptr, b, H, D, T - 1)
    B.pipo_dev_synchronize()
    a = o_ws.to_array(np.uint16, (b, H * D))
    n = o_na.to_array(np.uint16, (b, H * D))
    return q, kc, vc, a, n, ws_bytes


@pytest.mark.parametrize("first,second", [
    # (b, T, H, D): split shapes (few workgroups, long context), then a smaller one
    ((2, 2000, 8, 128), (1, 300, 4, 128)),
    ((1, 4000, 56, 128), (1, 700, 5, 128)),
    ((4, 1500, 12, 64), (3, 129, 6, 64)),
    ((3, 600, 56, 128), (1, 1, 2, 64)),
])
def test_noalloc_matches_workspace_entry_point(first, second):
    for k, (b, T, H, D) in enumerate((first, second)):
        log(f"attn_decode_noalloc call {k}: b={b} T={T} H={H} D={D}")
        q, kc, vc, a, n, ws_bytes = _both(b, T, H, D, seed=T * 7 + b + k)
        log(f"  workspace {ws_bytes} bytes")
        assert np.array_equal(a, n)
        got = n.view(np.float16).astype(np.float64)
        for i in range(b):
            want = causal_attention(q[i:i + 1].astype(np.float64), kc[:, i].astype(np.float64),
                                    vc[:, i].astype(np.float64), H)[0]
            assert np.abs(got[i] - want).max() <= 5e-3 * max(1.0, np.abs(want).max())


def test_noalloc_split_shapes_fit_the_array():
    """The largest split partials any shape needs stay below the 4 MiB array
    (the entry point would refuse a shape above it)."""
    worst = 0
    for D in (64, 128):
        for H in range(1, 129):
            for b in range(1, 65):
                worst = max(worst, B.pipo_op_attn_decode_workspace_bytes(b, H, D, 65535))
    assert 0 < worst <= 4 << 20
