"""CPU oracle for PIPO's decoder forward pass -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never uses it.

PIPO offloads weights and KV cache without changing the arithmetic: for fp16
or INT4 weights with fp16 activations (Section 4.1, "Workload") its result is
the plain decoder forward pass with greedy decoding.  The paper evaluates OPT
and LLaMA3.1 models (Section 4.1, "Model") and does not restate their
architectures, so this oracle writes out both decoders in their plain
definitions (the readings are listed in ``opt.py`` and ``llama.py``).
"""
from .opt import (  # noqa: F401
    OracleDecoder,
    causal_attention,
    dequant_int4_g64,
    layer_norm,
    param_count,
    layer_param_count,
    quant_kv_int4_g64,
    streamed_bytes_per_step,
)
from .llama import (  # noqa: F401
    LlamaDecoder,
    apply_rope,
    decoder_for,
    gqa_attention,
    llama_kv_bytes,
    llama_param_count,
    rms_norm,
    rope_frequencies,
    swiglu,
)
