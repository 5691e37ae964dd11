"""The pipeline schedule, checked on the CPU.

The library's engine executes the operation lists that pipo_sched_trace
returns.  Here those lists run on a simulated device: four in-order streams,
events with HIP semantics (a wait refers to the latest record issued before
it), random copy and kernel durations.  For every schedule variant the
simulated timeline must satisfy the orderings the pipeline relies on
(Algorithm 1 of the paper and its save-before-load rule, Section 3.2.2):

* a kernel starts only after every chunk of every tensor it reads has landed;
* a slot is refilled only after all kernels of its previous unit finished;
* with the KV cache in host memory, a layer's prefix is loaded only after the
  previous token's save of that layer completed, the save reads rows only
  after the QKV projection wrote them, and a KV buffer is overwritten only
  after its previous contents were read and saved;
* every tensor is streamed exactly once per pass, in full (also when a
  layer's matrices are copied as one merged range whose chunks span
  tensors).
"""
import itertools
import random
from collections import defaultdict

import pytest

from paper_2504_03664_amd import binding as B

COPY_H2D, COPY_D2H, WAIT, RECORD, KERNEL, DELAY, POISON, READBACK = range(8)
K_EMBED, K_LN1, K_QKV, K_ATTN, K_OPROJ, K_LN2, K_FC1, K_FC2, K_LNF, K_HEAD, K_ARGMAX = range(11)
SEG_MISC, SEG_WQKV, SEG_WQKV_SM, SEG_WO, SEG_WO_SM, SEG_W1, SEG_W1_SM, SEG_W2, SEG_W2_SM, SEG_HEAD = \
    range(10)
READS = {K_LN1: {SEG_MISC}, K_QKV: {SEG_MISC, SEG_WQKV, SEG_WQKV_SM},
         K_OPROJ: {SEG_MISC, SEG_WO, SEG_WO_SM}, K_LN2: {SEG_MISC},
         K_FC1: {SEG_MISC, SEG_W1, SEG_W1_SM}, K_FC2: {SEG_MISC, SEG_W2, SEG_W2_SM},
         K_HEAD: {SEG_HEAD}}
LAYER_KERNELS = [K_LN1, K_QKV, K_ATTN, K_OPROJ, K_LN2, K_FC1, K_FC2]


def make_config(n_layers, n_slots, n_h2d, layers_streamed, head_streamed, kv_on_host, w4,
                chunk, poison=False, delay=False, merged=False):
    cfg = B.PipoSchedConfig()
    cfg.n_layers, cfg.n_slots, cfg.n_h2d = n_layers, n_slots, n_h2d
    cfg.layers_streamed, cfg.head_streamed, cfg.kv_on_host = layers_streamed, head_streamed, kv_on_host
    cfg.poison, cfg.delay = poison, delay
    cfg.chunk_bytes = chunk
    seg = [0] * 10
    seg[SEG_MISC] = 13 * 1024
    for s, n in ((SEG_WQKV, 3), (SEG_WO, 1), (SEG_W1, 4), (SEG_W2, 4)):
        seg[s] = n * 65536 if not w4 else n * 16384
        if w4:
            seg[s + 1] = n * 2048
    off = 0
    for i in range(10):
        cfg.layer_seg_bytes[i] = seg[i]
        if i != SEG_HEAD:   # slot layout: segments at 4 KiB-aligned offsets
            cfg.layer_seg_off[i] = off
            off = (off + seg[i] + 4095) // 4096 * 4096
    cfg.merged = int(merged)
    cfg.head_bytes = 200 * 1024
    return cfg


def split_merged(cfg, c):
    """The per-segment pieces of a weight copy: a merged copy (named after
    segment 1, offset from its slot offset) covers every segment it
    overlaps; padding between segments belongs to none."""
    if not cfg.merged or c["layer"] < 0 or c["seg"] == SEG_MISC:
        return [c]
    base = cfg.layer_seg_off[SEG_WQKV]
    a0, a1 = c["off"], c["off"] + c["bytes"]
    pieces = []
    for seg in range(SEG_WQKV, SEG_HEAD):
        n = cfg.layer_seg_bytes[seg]
        lo = cfg.layer_seg_off[seg] - base
        x0, x1 = max(a0, lo), min(a1, lo + n)
        if n > 0 and x0 < x1:
            pieces.append(dict(c, seg=seg, off=x0 - lo, bytes=x1 - x0))
    return pieces


def parse(text):
    ops = []
    for line in text.strip().splitlines():
        v = [int(x) for x in line.split()]
        ops.append(dict(kind=v[0], stream=v[1], event=v[2], kernel=v[3], unit=v[4], layer=v[5],
                        slot=v[6], seg=v[7], kv=v[8], off=v[9], bytes=v[10]))
    return ops


def split_passes(ops):
    passes, cur = [], []
    for o in ops:
        cur.append(o)
        if o["kind"] == READBACK:
            passes.append(cur)
            cur = []
    assert not cur
    return passes


def simulate(passes, rng):
    """Assign [start, end) times to every op; returns the flat op list."""
    ready = [0.0] * 4
    last_record = {}
    host = 0.0
    flat = []
    for ops in passes:
        for o in ops:
            s = o["stream"]
            t0 = max(ready[s], host)
            if o["kind"] == WAIT:
                rec = last_record.get(o["event"])
                if rec is not None:
                    t0 = max(t0, rec["end"])
                dur = 0.0
            elif o["kind"] == RECORD:
                dur = 0.0
            elif o["kind"] in (COPY_H2D, COPY_D2H):
                dur = o["bytes"] / 65536 * rng.uniform(0.2, 3.0)
            elif o["kind"] == KERNEL:
                dur = rng.uniform(0.01, 2.0)
            elif o["kind"] in (DELAY, POISON):
                dur = rng.uniform(0.0, 1.0)
            else:  # readback
                dur = 0.01
            if rng.random() < 0.1:         # heavy tail: any op may stall
                dur *= 50.0
            o["start"], o["end"] = t0, t0 + dur
            ready[s] = o["end"]
            if o["kind"] == RECORD:
                last_record[o["event"]] = o
            flat.append(o)
        host = ops[-1]["end"]          # the host waits for the token readback
    return flat


def check(ops_by_pass, flat, cfg, pass_info, kv_row):
    eps = 1e-12
    kernels = [o for o in flat if o["kind"] == KERNEL]
    wcopies = [o for o in flat if o["kind"] == COPY_H2D and not o["kv"]]
    kvload = [o for o in flat if o["kind"] == COPY_H2D and o["kv"]]
    kvsave = [o for o in flat if o["kind"] == COPY_D2H]
    poisons = [o for o in flat if o["kind"] == POISON]
    copies_of = defaultdict(list)
    merged_of = defaultdict(list)
    for c in wcopies:
        for piece in split_merged(cfg, c):
            copies_of[(c["unit"], piece["seg"])].append(piece)
        if cfg.merged and c["layer"] >= 0 and c["seg"] != SEG_MISC:
            assert c["seg"] == SEG_WQKV
            merged_of[c["unit"]].append(c)
    # a merged range is copied once, in order-independent chunks of at most
    # chunk_bytes, from the first matrix to the end of the last
    last = max(s for s in range(SEG_WQKV, SEG_HEAD) if cfg.layer_seg_bytes[s] > 0)
    span = cfg.layer_seg_off[last] + cfg.layer_seg_bytes[last] - cfg.layer_seg_off[SEG_WQKV]
    for g, cs in merged_of.items():
        pos = 0
        for c in sorted(cs, key=lambda c: c["off"]):
            assert c["off"] == pos and 0 < c["bytes"] <= cfg.chunk_bytes
            pos += c["bytes"]
        assert pos == span

    # RAW on weights
    for k in kernels:
        if k["unit"] < 0:
            continue
        for seg in READS.get(k["kernel"], ()):
            for c in copies_of.get((k["unit"], seg), []):
                assert c["end"] <= k["start"] + eps, (k, c)
    # WAR on weight slots (copies and poison fills)
    by_slot = defaultdict(list)
    for k in kernels:
        if k["unit"] >= 0:
            by_slot[k["slot"]].append(k)
    for c in wcopies + [p for p in poisons if not p["kv"]]:
        for k in by_slot[c["slot"]]:
            if k["unit"] < c["unit"]:
                assert k["end"] <= c["start"] + eps, (c, k)
    for p in poisons:
        for c in (kvload if p["kv"] else wcopies):
            if c["unit"] == p["unit"]:
                assert c["start"] >= p["end"] - eps
    # every segment streamed once, in full, per unit instance
    for (g, seg), cs in copies_of.items():
        cs = sorted(cs, key=lambda c: c["off"])
        total = cfg.head_bytes if seg == SEG_HEAD else cfg.layer_seg_bytes[seg]
        pos = 0
        for c in cs:
            assert c["off"] == pos and c["bytes"] <= cfg.chunk_bytes
            pos += c["bytes"]
        assert pos == total
    n_units = (cfg.n_layers if cfg.layers_streamed else 0) + (1 if cfg.head_streamed else 0)
    units = {g for (g, _) in copies_of}
    assert units == set(range(len(units)))
    assert len(units) >= n_units * len(ops_by_pass)
    # each pass computes every layer in order, then the head
    for ops in ops_by_pass:
        ks = [o["kernel"] for o in ops if o["kind"] == KERNEL]
        assert ks == [K_EMBED] + LAYER_KERNELS * cfg.n_layers + [K_LNF, K_HEAD, K_ARGMAX]

    if not cfg.kv_on_host:
        assert not kvload and not kvsave
        return
    qkv = {k["unit"]: k for k in kernels if k["kernel"] == K_QKV}
    attn = {k["unit"]: k for k in kernels if k["kernel"] == K_ATTN}
    loads, saves = defaultdict(list), defaultdict(list)
    for c in kvload:
        loads[c["unit"]].append(c)
    for c in kvsave:
        saves[c["unit"]].append(c)
    for g, a in attn.items():
        for c in loads[g]:
            assert c["end"] <= qkv[g]["start"] + eps
        assert qkv[g]["end"] <= a["start"] + eps
        assert len(saves[g]) == 2
        for c in saves[g]:
            assert c["start"] >= qkv[g]["end"] - eps
    slot_of = {g: a["slot"] for g, a in attn.items()}
    for g2 in attn:
        for g1 in attn:
            if g1 >= g2 or slot_of[g1] != slot_of[g2]:
                continue
            readers_end = max([attn[g1]["end"]] + [c["end"] for c in saves[g1]])
            for c in loads[g2]:
                assert c["start"] >= readers_end - eps
            assert qkv[g2]["start"] >= readers_end - eps
    # host KV: the save of layer j at an earlier pass completes before any later load of j
    layer_of = {g: a["layer"] for g, a in attn.items()}
    for g2, cs in loads.items():
        for g1, ss in saves.items():
            if g1 < g2 and layer_of[g1] == layer_of[g2]:
                for c in cs:
                    for s in ss:
                        assert c["start"] >= s["end"] - eps
    # bytes: loads cover the prefix, saves the new rows
    for pi, (ops, info) in enumerate(zip(ops_by_pass, pass_info)):
        prefill, pos0, T = info
        for o in ops:
            if o["kind"] == COPY_D2H:
                assert o["off"] == pos0 * kv_row and o["bytes"] == T * kv_row
        got = defaultdict(int)
        for o in ops:
            if o["kind"] == COPY_H2D and o["kv"]:
                got[(o["unit"], o["seg"])] += o["bytes"]
        if prefill:
            assert not got
        else:
            assert got and all(v == pos0 * kv_row for v in got.values())


VARIANTS = list(itertools.product(
    [1, 3],            # layers
    [1, 2, 3, 4],      # slots (1: the memory-efficient pipeline)
    [1, 2],            # h2d streams
    [(1, 1, 0), (1, 0, 0), (0, 1, 0), (1, 1, 1), (1, 0, 1)],  # layers/head streamed, kv on host
    [False, True],     # int4 segments
    [False, True],     # merged copies of a layer's matrices
))


@pytest.mark.parametrize("L,S,nh,mode,w4,merged", VARIANTS)
def test_schedule_orderings(L, S, nh, mode, w4, merged):
    ls, hs, kvh = mode
    rng = random.Random(hash((L, S, nh, mode, w4, merged)) & 0xFFFF)
    P, G = 5, 4
    passes = [(True, 0, P)] + [(False, P + i, 1) for i in range(G)] + \
             [(True, 0, 3)] + [(False, 3, 1)]
    kv_row = 4096
    for chunk in (32 * 1024, 50 * 1024, 1 << 30):
        cfg = make_config(L, S, nh, ls, hs, kvh, w4, chunk, poison=(chunk < 1 << 30),
                          delay=(nh == 2), merged=merged)
        text = B.pipo_sched_trace(cfg, passes, kv_row_bytes=kv_row)
        for trial in range(6):
            ops_by_pass = split_passes(parse(text))
            assert len(ops_by_pass) == len(passes)
            flat = simulate(ops_by_pass, rng)
            check(ops_by_pass, flat, cfg, passes, kv_row)


def test_lookahead_keeps_link_busy_across_steps():
    """With fast kernels, the copy stream never waits for the host between
    decode steps: the next step's first units are already queued."""
    cfg = make_config(4, 3, 1, 1, 1, 0, False, 1 << 30)
    passes = [(True, 0, 4)] + [(False, 4 + i, 1) for i in range(6)]
    ops_by_pass = split_passes(parse(B.pipo_sched_trace(cfg, passes)))
    # copies of pass i+1's first two units are issued inside pass i
    for i in range(len(passes) - 1):
        units_in_pass = {o["unit"] for o in ops_by_pass[i] if o["kind"] == KERNEL and o["unit"] >= 0}
        issued = {o["unit"] for o in ops_by_pass[i] if o["kind"] == COPY_H2D}
        assert max(issued) == max(units_in_pass) + 2


def test_invalid_config_rejected():
    for bad in (make_config(2, 0, 1, 1, 1, 0, False, 4096),
                make_config(2, 2, 3, 1, 1, 0, False, 4096),
                make_config(0, 2, 1, 1, 1, 0, False, 4096)):
        with pytest.raises(ValueError):
            B.pipo_sched_trace(bad, [(True, 0, 2)])
