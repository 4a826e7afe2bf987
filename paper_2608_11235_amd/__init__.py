"""MI355X (gfx950) hot path of CORA-Diff: one blockwise masked-diffusion denoising step.

The work runs in ``libcora.so`` (hand-written HIP kernels behind the C ABI in
``include/cora.h``); this package is the thin Python binding over it.  torch
supplies device memory and the HIP stream only.

    Model(cfg, seed, max_batch, max_seq)   seeded weights + workspace
    Model.forward_logits(tokens, row_begin, n_rows)
    Model.denoise_step(state, sched, gate)
    Model.block_decode(prompt, gen_len, sched, gate)
    vocab_gate(logits, ...)                 the vocab/gate kernel alone
"""
from .api import (  # noqa: F401
    Model, DecodeState, Sched, Gate, vocab_gate, vocab_gate_noalloc, model_cfg_from,
    TENSOR_EMBED, TENSOR_LM_HEAD, layer_tensor_id,
)
from .configs import TINY, LLADA_8B, DREAM_7B, ModelConfig  # noqa: F401
