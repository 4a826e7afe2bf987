"""Seeded prompts, decode states and the vocab/gate logits workload."""
from dataclasses import dataclass

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (round to nearest even), returned as uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def prompt_tokens(seed: int, batch: int, prompt_len: int, vocab: int, mask_id: int) -> np.ndarray:
    """Uniform tokens over [0, vocab) without the mask id; int32 [batch, prompt_len]."""
    rng = np.random.Generator(np.random.PCG64(seed))
    t = rng.integers(0, vocab - 1, size=(batch, prompt_len), dtype=np.int64)
    t = t + (t >= mask_id)
    return t.astype(np.int32)


def initial_decode_state(prompt: np.ndarray, gen_len: int, mask_id: int) -> dict:
    """Canvas = prompt followed by gen_len mask tokens; all generation positions unresolved."""
    B, P = prompt.shape
    L = P + gen_len
    tokens = np.full((B, L), mask_id, dtype=np.int32)
    tokens[:, :P] = prompt
    unresolved = np.zeros((B, L), dtype=np.uint8)
    unresolved[:, P:] = 1
    return {
        "tokens": tokens,
        "unresolved": unresolved,
        "prev_top1": np.full((B, L), -1, dtype=np.int32),
        "persist": np.zeros((B, L), dtype=np.int32),
        "block_idx": np.zeros(B, dtype=np.int32),
        "step_idx": np.zeros(B, dtype=np.int32),
    }


@dataclass
class VocabGateWorkload:
    logits_bits: np.ndarray   # uint16 [B, L, V] bf16 bits, one row per canvas position
    spike_token: np.ndarray   # int64 [B, L]
    state: dict               # decode state arrays (see initial_decode_state)
    prompt_len: int
    block_len: int
    steps_per_block: int
    vocab: int
    mask_id: int

    @property
    def shape(self):
        return self.logits_bits.shape


def vocab_gate_workload(seed: int = 2, batch: int = 8, prompt_len: int = 256, gen_len: int = 256,
                        vocab: int = 126464, mask_id: int = 126336, block_len: int = 32,
                        steps_per_block: int = 32, masked_in_block: int = 8,
                        spike_max: float = 12.0) -> VocabGateWorkload:
    """bf16 logits [B, L, V] ~ N(0,1) plus one spike of height U(0, spike_max) at a uniform
    token per row, with a mid-block decode state: each batch row has a seeded active
    generation block holding `masked_in_block` masked positions, earlier blocks resolved
    and later blocks masked."""
    rng = np.random.Generator(np.random.PCG64(seed))
    L = prompt_len + gen_len
    n_blocks = gen_len // block_len
    bits = np.empty((batch, L, vocab), dtype=np.uint16)
    spike_tok = rng.integers(0, vocab, size=(batch, L))
    spike_h = rng.uniform(0.0, spike_max, size=(batch, L)).astype(np.float32)
    for b in range(batch):
        x = rng.standard_normal((L, vocab), dtype=np.float32)
        x[np.arange(L), spike_tok[b]] += spike_h[b]
        bits[b] = f32_to_bf16_bits(x)

    tokens = rng.integers(0, vocab - 1, size=(batch, L), dtype=np.int64)
    tokens = (tokens + (tokens >= mask_id)).astype(np.int32)
    unresolved = np.zeros((batch, L), dtype=np.uint8)
    block_idx = rng.integers(0, n_blocks, size=batch).astype(np.int32)
    step_idx = rng.integers(1, steps_per_block, size=batch).astype(np.int32)
    for b in range(batch):
        lo = prompt_len + int(block_idx[b]) * block_len
        masked = lo + rng.choice(block_len, size=masked_in_block, replace=False)
        unresolved[b, masked] = 1
        unresolved[b, lo + block_len:] = 1
    tokens[unresolved == 1] = mask_id
    keep_spike = rng.random((batch, L)) < 0.5
    rand_tok = rng.integers(0, vocab, size=(batch, L))
    prev = np.where(keep_spike, spike_tok, rand_tok).astype(np.int32)
    persist = rng.integers(0, 4, size=(batch, L)).astype(np.int32)
    state = {
        "tokens": tokens, "unresolved": unresolved, "prev_top1": prev, "persist": persist,
        "block_idx": block_idx, "step_idx": step_idx,
    }
    return VocabGateWorkload(bits, spike_tok, state, prompt_len, block_len, steps_per_block,
                             vocab, mask_id)
