"""Pins of the seeded input generators (weights, prompts, vocab/gate workload)."""
import json
import os

import numpy as np
import pytest
import torch
from scipy import stats

import seeded_inputs as si
from seeded_inputs.workloads import bf16_bits_to_f32, f32_to_bf16_bits


def test_splitmix64_published_vectors(golden_dir):
    with open(os.path.join(golden_dir, "splitmix64_vectors.json")) as f:
        g = json.load(f)
    got = si.splitmix64_stream(g["seed"], len(g["outputs"]))
    assert [str(int(x)) for x in got] == g["outputs"]


def test_weight_generator_is_normal_0_02():
    w = si.gen_tensor(0, 7, (400_000,))
    assert abs(w.mean()) < 3 * 0.02 / np.sqrt(w.size) * 2
    assert w.std() == pytest.approx(0.02, rel=0.01)
    ks = stats.kstest(w / 0.02, "norm")
    assert ks.pvalue > 1e-3


def test_weight_generator_counter_based():
    full = si.gen_tensor(5, 101, (64, 48), as_bits=True)
    part = si.gen_elements(5, 101, 17 * 48 + 3, 100, 0.02)
    assert (full.reshape(-1)[17 * 48 + 3: 17 * 48 + 103] == part).all()
    rows = si.gen_rows(5, 101, [60, 2, 2], 48)
    np.testing.assert_array_equal(rows, bf16_bits_to_f32(full[[60, 2, 2]]))
    other = si.gen_tensor(5, 102, (64, 48), as_bits=True)
    assert (other != full).mean() > 0.9
    other_seed = si.gen_tensor(6, 101, (64, 48), as_bits=True)
    assert (other_seed != full).mean() > 0.9


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).normal(0, 3, 100_000).astype(np.float32)
    x[:4] = [1.00390625, 1.01171875, -2.0078125, 0.0]   # exact halfway cases
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert (f32_to_bf16_bits(x) == want).all()


def test_prompt_tokens_exclude_mask():
    t = si.prompt_tokens(1, 4, 5000, 50, 17)
    assert t.dtype == np.int32 and (t != 17).all() and t.min() >= 0 and t.max() == 49
    assert len(np.unique(t)) == 49


def test_vocab_gate_workload_layout():
    w = si.vocab_gate_workload(seed=2, batch=3, prompt_len=16, gen_len=64, vocab=300,
                               mask_id=290, block_len=32, masked_in_block=8)
    st = w.state
    B, L, V = w.shape
    assert (B, L, V) == (3, 80, 300)
    for b in range(B):
        lo = 16 + 32 * int(st["block_idx"][b])
        assert st["unresolved"][b, lo:lo + 32].sum() == 8
        assert st["unresolved"][b, :lo].sum() == 0
        assert (st["unresolved"][b, lo + 32:] == 1).all()
        assert ((st["tokens"][b] == 290) == (st["unresolved"][b] == 1)).all()
    assert (st["step_idx"] >= 1).all()
    x = bf16_bits_to_f32(w.logits_bits)
    # the spike sits on the drawn token
    hit = np.take_along_axis(x, w.spike_token[..., None], -1)[..., 0]
    assert (hit > x.mean(-1)).mean() > 0.9
