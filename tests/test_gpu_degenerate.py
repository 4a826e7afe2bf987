"""Degenerate decode shapes through the C ABI: an empty prompt, one-position blocks, the
largest block (256 positions), and a short canvas that is neither a multiple of 64 nor of
4.  They are checked by properties that hold at any size: with the gate off every block
takes exactly its dense number of passes (S_b); no mask is left at the end; the prompt is
untouched; cora_block_decode equals the step-by-step trajectory of cora_denoise_step; and
with one-position blocks (one transfer per step) each committed token is the lowest-id
argmax, mask id left out, of the logits the same model gives that row at that step."""
import numpy as np
import pytest

import seeded_inputs as si
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import bf16_to_f32

pytestmark = pytest.mark.gpu

SPEC = si.TINY


def _stepwise(m, prompt, P, G, blk, steps, gate):
    from paper_2608_11235_amd import DecodeState, Sched
    host = si.initial_decode_state(prompt, G, SPEC.mask_id)
    st = DecodeState.from_host(host, P, G, blk, blk)
    sched = Sched(blk, steps)
    n_blocks = G // blk
    for _ in range(n_blocks * steps):
        if (st.to_host()["block_idx"] >= n_blocks).all():
            break
        m.denoise_step(st, sched, gate)
    return st.to_host()


@pytest.mark.parametrize("P,G,blk,steps,gate_on", [
    (0, 64, 32, 16, False),     # empty prompt: the canvas starts all masks
    (0, 64, 32, 16, True),
    (16, 256, 256, 32, False),  # the largest block: 256 positions, k = 8 per step
    (5, 32, 8, 4, True),        # L = 37: padded key tiles and a ragged row group
    (16, 8, 1, 1, True),        # one-position blocks: one transfer per step
])
def test_degenerate_decode(P, G, blk, steps, gate_on):
    require_gpu()
    from paper_2608_11235_amd import Gate, Model, Sched
    B, L = 2, P + G
    log_case(f"degenerate decode P={P} G={G} blk={blk} S={steps} gate={gate_on}")
    prompt = si.prompt_tokens(9, B, max(P, 1), SPEC.vocab, SPEC.mask_id)[:, :P]
    gate = Gate(0.65, 1, gate_on)
    with Model(SPEC, seed=0, max_batch=B, max_seq=L) as m:
        final = _stepwise(m, prompt, P, G, blk, steps, gate)
        out, passes, total = m.block_decode(to_dev(np.ascontiguousarray(prompt)), G,
                                            Sched(blk, steps), gate)
    out = out.cpu().numpy()
    assert (out == final["tokens"]).all(), "block_decode != step-by-step"
    assert (passes == final["passes"]).all()
    assert (out[:, :P] == prompt).all()
    assert (out[:, P:] != SPEC.mask_id).all()
    if not gate_on:
        assert (passes == steps).all() and total == (G // blk) * steps
    assert (passes >= 1).all() and (passes <= steps).all()


def test_one_position_blocks_commit_the_argmax():
    """blk = 1, S = 1: every step commits its single position, and the token is the
    lowest-id argmax (mask id left out) of the model's logits for that row of the canvas
    the step saw."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    B, P, G = 2, 16, 8
    L = P + G
    log_case("one-position blocks: committed token == argmax of own logits")
    prompt = si.prompt_tokens(10, B, P, SPEC.vocab, SPEC.mask_id)
    host = si.initial_decode_state(prompt, G, SPEC.mask_id)
    with Model(SPEC, seed=0, max_batch=B, max_seq=L) as m:
        st = DecodeState.from_host(host, P, G, 1, 1)
        for j in range(G):
            pre = st.to_host()
            lg = bf16_to_f32(m.forward_logits(to_dev(pre["tokens"]), P + j, 1).cpu().numpy())
            m.denoise_step(st, Sched(1, 1), Gate(0.65, 1, True))
            post = st.to_host()
            x = lg[:, 0].astype(np.float64)
            x[:, SPEC.mask_id] = -np.inf
            want = np.argmax(x, axis=-1)
            assert (post["tokens"][:, P + j] == want).all(), f"step {j}"
            assert (post["unresolved"][:, P + j] == 0).all()
            assert (post["passes"][:, j] == 1).all()
