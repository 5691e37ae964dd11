"""Memory planning and the automatic configuration (Section 3.5, Eq. (1)):
host-side computations of the library, no GPU needed.  The byte counts are
checked against the oracle's independent accounting, the choice against a
brute force over every placement and pipeline."""
import itertools

import pytest

import synth
from oracle import layer_param_count, streamed_bytes_per_step
from paper_2504_03664_amd import binding as B
from paper_2504_03664_amd.model import c_policy, c_shape

GB = 10 ** 9
OPT30 = synth.OPT_30B


def plan(shape, **pol):
    return B.pipo_plan_policy(c_shape(shape), c_policy(**pol))


@pytest.mark.parametrize("shape,wfmt,kv_fmt,b,s", [
    (synth.OPT_6_7B, "fp16", "fp16", 16, 544),
    (synth.OPT_13B, "int4", "fp16", 32, 544),
    (OPT30, "int4", "int4", 128, 544),
    (synth.OPT_125M, "fp16", "fp16", 4, 40),
])
def test_step_bytes_match_oracle_accounting(shape, wfmt, kv_fmt, b, s):
    """Streamed bytes per step = the oracle's closed form (weights, head and
    the KV prefix) + token ids and embedding rows + the padding of each
    layer's small-tensor copy to 32 KiB (shorter copies would run on a blit
    kernel instead of a DMA engine)."""
    d = shape.d_model
    small = layer_param_count(d, shape.d_ffn) - (4 * d * d + 2 * d * shape.d_ffn)
    extra = b * 4 + b * d * 2 + shape.n_layers * max(0, 32768 - 2 * small)
    p = plan(shape, wfmt=wfmt, kv_fmt=kv_fmt, max_batch=b, max_seq=s)
    want = streamed_bytes_per_step(shape.n_layers, d, shape.d_ffn, shape.vocab, wfmt)
    assert p["h2d_bytes_per_step"] == want + extra
    p = plan(shape, wfmt=wfmt, kv_fmt=kv_fmt, kv_on_host=True, max_batch=b, max_seq=s)
    want = streamed_bytes_per_step(shape.n_layers, d, shape.d_ffn, shape.vocab, wfmt,
                                   kv_batch=b, kv_len=s - 1, kv_fmt=kv_fmt)
    assert p["h2d_bytes_per_step"] == want + extra
    # nothing streamed but the token ids when everything is resident
    p = plan(shape, wfmt=wfmt, kv_fmt=kv_fmt, weights_on_host=False, embed_on_host=False,
             max_batch=b, max_seq=s)
    assert p["h2d_bytes_per_step"] == b * 4


def test_plan_kv_bytes_and_pipeline():
    b, s = 64, 544
    p = plan(OPT30, max_batch=b, max_seq=s)
    assert p["kv_bytes"] == OPT30.n_layers * 2 * b * s * OPT30.d_model * 2   # C of Section 3.5
    assert p["pipeline"] == B.PIPO_PIPE_PERFORMANCE
    p1 = plan(OPT30, max_batch=b, max_seq=s, n_weight_slots=1, kv_on_host=True)
    assert p1["pipeline"] == B.PIPO_PIPE_MEMORY_EFFICIENT
    assert p1["hbm_bytes"] < p["hbm_bytes"] and p1["host_kv_bytes"] >= p["kv_bytes"]
    # one slot less saves exactly one layer unit and one KV buffer pair
    p2 = plan(OPT30, max_batch=b, max_seq=s, n_weight_slots=2, kv_on_host=True)
    p3 = plan(OPT30, max_batch=b, max_seq=s, n_weight_slots=3, kv_on_host=True)
    assert p3["hbm_bytes"] - p2["hbm_bytes"] == p2["hbm_bytes"] - p1["hbm_bytes"] > 0


def candidates(shape, wfmt, kv_fmt, b, s):
    for w, e, k, n in itertools.product((0, 1), (0, 1), (0, 1), (3, 2, 1)):
        if k > w or (not w and not e and n != 3):
            continue
        yield dict(weights_on_host=bool(w), embed_on_host=bool(e), kv_on_host=bool(k),
                   n_weight_slots=n), plan(shape, wfmt=wfmt, kv_fmt=kv_fmt, max_batch=b, max_seq=s,
                                           weights_on_host=bool(w), embed_on_host=bool(e),
                                           kv_on_host=bool(k), n_weight_slots=n)


@pytest.mark.parametrize("hbm_gb", [288, 120, 80, 24, 12, 8])
@pytest.mark.parametrize("wfmt,kv_fmt", [("fp16", "fp16"), ("int4", "int4")])
def test_configure_is_the_best_feasible_choice(hbm_gb, wfmt, kv_fmt):
    b, s, host = 64, 544, 512 * GB
    pol, p = B.pipo_configure(c_shape(OPT30), 0 if wfmt == "fp16" else 1,
                              0 if kv_fmt == "fp16" else 1, b, s, hbm_gb * GB, host)
    assert p["hbm_bytes"] <= hbm_gb * GB and pol.hbm_budget_bytes == hbm_gb * GB
    feasible = [(c, q) for c, q in candidates(OPT30, wfmt, kv_fmt, b, s)
                if q["hbm_bytes"] <= hbm_gb * GB and q["host_kv_bytes"] <= host]
    best = min(q["h2d_bytes_per_step"] for _, q in feasible)
    assert p["h2d_bytes_per_step"] == best
    slots = max(c["n_weight_slots"] for c, q in feasible if q["h2d_bytes_per_step"] == best)
    assert pol.n_weight_slots == slots or (not pol.weights_on_host and not pol.embed_on_host)
    assert p == B.pipo_plan_policy(c_shape(OPT30), pol)


def test_configure_follows_eq1_on_the_30b_shape():
    """Eq. (1): weights in HBM when everything fits; streamed from host memory
    otherwise; the performance-optimized pipeline while its memory fits, the
    memory-efficient one below that; nothing below the single-layer minimum."""
    b, s, host = 64, 544, 512 * GB
    conf = lambda hbm: B.pipo_configure(c_shape(OPT30), 0, 0, b, s, hbm, host)  # noqa: E731
    pol, p = conf(288 * GB)
    assert not pol.weights_on_host and not pol.embed_on_host and not pol.kv_on_host
    pol, p = conf(80 * GB)                          # weights 60 GB + KV 48 GB do not fit
    assert pol.weights_on_host and not pol.kv_on_host and pol.n_weight_slots == 3
    pol, p = conf(24 * GB)                          # the KV cache goes to host memory
    assert pol.weights_on_host and pol.kv_on_host and p["pipeline"] == B.PIPO_PIPE_PERFORMANCE
    pol, p = conf(8 * GB)
    assert pol.kv_on_host and p["pipeline"] == B.PIPO_PIPE_MEMORY_EFFICIENT
    with pytest.raises(B.PipoError) as e:
        conf(4 * GB)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_OOM_DEVICE"
    with pytest.raises(B.PipoError) as e:           # KV fits neither in HBM nor on the host
        B.pipo_configure(c_shape(OPT30), 0, 0, b, s, 24 * GB, 10 * GB)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_OOM_HOST"


def test_more_memory_never_streams_more():
    b, s, host = 32, 544, 512 * GB
    last = None
    for hbm_gb in (6, 8, 12, 16, 24, 32, 48, 64, 96, 128, 200, 288):
        try:
            _, p = B.pipo_configure(c_shape(synth.OPT_13B), 1, 0, b, s, hbm_gb * GB, host)
        except B.PipoError:
            assert last is None
            continue
        if last is not None:
            assert p["h2d_bytes_per_step"] <= last
        last = p["h2d_bytes_per_step"]
    assert last == b * 4


def test_disk_tier_plan():
    """The disk tier's file holds every layer unit (slot layout); a step reads
    it once; the layers leave host memory, the head and the staging ring
    stay; the link carries the same bytes as from host memory."""
    b, s = 64, 544
    host = plan(OPT30, max_batch=b, max_seq=s)
    disk = plan(OPT30, max_batch=b, max_seq=s, weights_on_disk=True)
    L, d, F, V = OPT30.n_layers, OPT30.d_model, OPT30.d_ffn, OPT30.vocab
    layer_copy = (12 * d * d + 13 * d) * 2                       # fp16 tensors of a layer
    assert disk["disk_bytes"] == disk["disk_bytes_per_step"]
    assert 0 <= disk["disk_bytes"] - L * layer_copy < L * 5 * 4096   # 4 KiB-aligned segments
    assert disk["h2d_bytes_per_step"] == host["h2d_bytes_per_step"]
    ring = (16 + 1) * (64 << 20)                      # pinned ring + the direct-I/O chunk
    assert host["host_weight_bytes"] == L * layer_copy + V * d * 2
    assert disk["host_weight_bytes"] == V * d * 2 + ring
    assert disk["hbm_bytes"] == host["hbm_bytes"] and host["disk_bytes"] == 0
    with pytest.raises(B.PipoError) as e:
        plan(OPT30, max_batch=b, max_seq=s, weights_on_host=False, weights_on_disk=True)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_UNSUPPORTED"


def test_configure_puts_the_layers_on_disk_only_when_host_memory_is_short():
    """Eq. (1)'s third tier: weights that fit neither in HBM nor in host
    memory go to disk; with enough host memory the disk is not used."""
    b, s = 64, 544
    conf = lambda host, disk: B.pipo_configure(c_shape(OPT30), 0, 0, b, s, 80 * GB, host,  # noqa: E731
                                               disk)
    pol, p = conf(512 * GB, 200 * GB)
    assert pol.weights_on_host and not pol.weights_on_disk and p["disk_bytes"] == 0
    pol, p = conf(16 * GB, 200 * GB)                 # 60 GB of layers do not fit on the host
    assert pol.weights_on_disk and p["disk_bytes"] > 0
    assert p["host_weight_bytes"] + p["host_kv_bytes"] <= 16 * GB
    with pytest.raises(B.PipoError) as e:            # no room on disk either
        conf(16 * GB, 30 * GB)
    assert B.STATUS_NAMES[e.value.status] == "PIPO_ERR_OOM_HOST"
