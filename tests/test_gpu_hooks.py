"""The measurement and bookkeeping hooks of the C ABI on the GPU.

cora_model_set_timing / read_timing: every gate/up GEMM launch of a timed pass is counted
once (one per layer per pass), the summed event time is positive and plausible, reading
clears both figures, untimed passes add nothing, and stamping the launches changes no
result (same tokens and state, bit for bit, as an untimed run).
cora_model_device_bytes: the weight bytes cover at least every bf16 weight matrix of the
spec and do not depend on the workspace size, which grows with the canvas."""
import numpy as np
import pytest

import seeded_inputs as si
from tests.gpu_common import log_case, require_gpu

pytestmark = pytest.mark.gpu

SPEC = si.TINY
B, P, G, BLK, STEPS = 2, 16, 32, 16, 8


def _run(m, n_timed, n_untimed):
    from paper_2608_11235_amd import DecodeState, Gate, Sched
    prompt = si.prompt_tokens(21, B, P, SPEC.vocab, SPEC.mask_id)
    st = DecodeState.from_host(si.initial_decode_state(prompt, G, SPEC.mask_id), P, G, BLK, BLK)
    sched, gate = Sched(BLK, STEPS), Gate(0.65, 1, True)
    m.set_timing(True)
    for _ in range(n_timed):
        m.denoise_step(st, sched, gate)
    m.set_timing(False)
    for _ in range(n_untimed):
        m.denoise_step(st, sched, gate)
    return st.to_host()


def test_timing_counts_each_gate_up_launch_and_changes_nothing():
    require_gpu()
    from paper_2608_11235_amd import Model
    log_case("timing hooks: launch count, clearing, results unchanged")
    with Model(SPEC, seed=0, max_batch=B, max_seq=P + G) as m:
        assert m.read_timing() == (0.0, 0)
        timed = _run(m, 3, 2)
        ms, n = m.read_timing()
        assert n == 3 * SPEC.n_layers
        assert 0.0 < ms < 10.0 * n          # each launch took more than 0 and under 10 ms
        assert m.read_timing() == (0.0, 0)  # reading cleared both figures
    with Model(SPEC, seed=0, max_batch=B, max_seq=P + G) as m:
        plain = _run(m, 0, 5)
        assert m.read_timing() == (0.0, 0)
    for key in plain:
        assert np.array_equal(timed[key], plain[key]), key


def test_device_bytes():
    require_gpu()
    from paper_2608_11235_amd import Model
    log_case("device bytes: weights cover the spec, workspace grows with the canvas")
    d, V, hd = SPEC.d_model, SPEC.vocab, SPEC.head_dim
    f_pad = -(-SPEC.ffn_dim // 64) * 64
    qkv_n = (SPEC.n_heads + 2 * SPEC.n_kv_heads) * hd
    per_layer = qkv_n * d + d * SPEC.n_heads * hd + 2 * f_pad * d + d * f_pad
    matrices = 2 * (2 * V * d + SPEC.n_layers * per_layer)  # bf16 embed, LM head, layers
    with Model(SPEC, seed=0, max_batch=B, max_seq=64) as m:
        w1, ws1 = m.device_bytes()
    with Model(SPEC, seed=0, max_batch=B, max_seq=256) as m:
        w2, ws2 = m.device_bytes()
    assert matrices <= w1 <= 3 * matrices
    assert w2 == w1
    assert 0 < ws1 < ws2


def test_binding_refuses_misread_tensors():
    require_gpu()
    import torch
    from paper_2608_11235_amd import Model
    log_case("binding: wrong dtype, non-contiguous and undersized tensors refused")
    with Model(SPEC, seed=0, max_batch=B, max_seq=P + G) as m:
        tok = torch.zeros((B, P + G), dtype=torch.int32, device="cuda")
        with pytest.raises(TypeError):
            m.forward_logits(tok.long(), 0, 4)
        with pytest.raises(ValueError, match="contiguous"):
            m.forward_logits(torch.zeros((P + G, B), dtype=torch.int32, device="cuda").t(), 0, 4)
        small = torch.empty((B, 3, SPEC.vocab), dtype=torch.int16, device="cuda")
        with pytest.raises(ValueError, match="elements"):
            m.forward_logits(tok, 0, 4, out=small)
        m.forward_logits(tok, 0, 3, out=small)   # the right size goes through
        torch.cuda.synchronize()
