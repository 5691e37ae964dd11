"""The stored full-batch oracle results (``tests/golden/fullbatch``) are
the oracle's own: every case of the writer's table is stored, its metadata
and shapes match the table and the workload, and one row of the two-layer
slices recomputed here by the oracle gives the stored values.  (The GPU
comparison itself is in ``test_gpu_fullbatch.py``.)"""
import json
import os
import sys

import numpy as np
import pytest

import synth
from oracle import decoder_for

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "golden"))
import make_fullbatch as MF  # noqa: E402


def load(name):
    with np.load(os.path.join(MF.OUT_DIR, name + ".npz"), allow_pickle=False) as z:
        fx = {k: z[k] for k in z.files}
    fx["meta"] = json.loads(str(fx["meta"]))
    return fx


@pytest.mark.parametrize("name", sorted(MF.CASES))
def test_stored_case_matches_the_table(name):
    case = MF.CASES[name]
    fx = load(name)
    m = fx["meta"]
    wl = synth.WORKLOADS[case["widx"]]
    R = wl.batch if case.get("rows") is None else case["rows"]
    assert m["case"] == name and m["workload"] == wl.name and m["stream"] == case["widx"]
    assert m["writer"] == "tests/golden/make_fullbatch.py"
    assert m["reading"] == case.get("reading", "fp32")
    assert m["layers"] == (case.get("layers") or wl.shape.n_layers)
    assert m["kv_int4"] == (wl.kv_fmt == "int4") and m["zero_kv"] == bool(case.get("zero_kv"))
    assert m["weight_seed"] == synth.DEFAULT_SEED
    assert np.array_equal(fx["rows"], np.arange(R))
    assert fx["top_idx"].shape == fx["top_val"].shape == (R, wl.gen, MF.TOP)
    assert fx["absmax"].shape == (R, wl.gen)
    assert np.array_equal(fx["samp_idx"], MF.sampled_ids(case["widx"], wl.shape.vocab))
    assert fx["samp_val"].shape == (R, wl.gen, MF.N_SAMPLED)
    tv = fx["top_val"].astype(np.float64)
    assert np.all(np.diff(tv, axis=-1) <= 0)                  # largest first
    assert np.all(np.abs(tv) <= fx["absmax"][..., None] * (1 + 1e-6))
    assert np.all((fx["top_idx"] >= 0) & (fx["top_idx"] < wl.shape.vocab))


@pytest.mark.parametrize("name", ["opt-6.7b-l2", "llama3.1-8b-int4-l2"])
def test_one_row_recomputed_by_the_oracle(name):
    case = MF.CASES[name]
    fx = load(name)
    wl, shape, model, prompt, forced, rows = MF.case_inputs(case)
    tokens = np.concatenate([prompt[:1], forced[:1]], axis=1)
    dec = decoder_for(model, np.float32, kv_int4=wl.kv_fmt == "int4",
                      fp16_operands=case.get("reading") == "fp16ops")
    lg = dec.forward(tokens, last=wl.gen)[0].astype(np.float64)   # [gen][V]
    scale = fx["absmax"][0].astype(np.float64)
    got_top = np.take_along_axis(lg, fx["top_idx"][0].astype(np.int64), axis=-1)
    assert np.allclose(got_top, fx["top_val"][0], rtol=0, atol=1e-5 * scale.max())
    assert np.allclose(lg[:, fx["samp_idx"]], fx["samp_val"][0], rtol=0, atol=1e-5 * scale.max())
    assert np.allclose(np.abs(lg).max(-1), scale, rtol=1e-5)
    # the stored greedy token is the recomputed one, up to a near tie
    best = lg.argmax(-1)
    stored = fx["top_idx"][0, :, 0]
    gap = lg[np.arange(len(best)), best] - lg[np.arange(len(best)), stored]
    assert np.all((best == stored) | (gap <= 1e-5 * scale))
