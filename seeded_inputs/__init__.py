"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This package holds no step of the decoding method.  It produces

* the workload shapes (the tiny model, the LLaDA-8B and Dream-7B shapes),
* model weights from a counter-based generator (host half; the GPU library
  implements the same definition on its own, see ``wgen.c``),
* prompts, and the vocab/gate workload (logits plus decode state).

Everything is a pure function of its seed.
"""
from .spec import (  # noqa: F401
    ModelSpec, TINY, LLADA_8B, DREAM_7B, TENSOR_EMBED, TENSOR_LM_HEAD,
    layer_tensor_id, LAYER_TENSORS,
)
from .weights import (  # noqa: F401
    gen_tensor, gen_rows, gen_elements, splitmix64_stream, gen_layer, HostWeights,
)
from .workloads import (  # noqa: F401
    prompt_tokens, vocab_gate_workload, VocabGateWorkload, initial_decode_state,
)
