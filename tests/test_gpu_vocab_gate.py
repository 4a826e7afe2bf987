"""GPU parity of the vocab/gate kernel alone on shared bf16 logits.

Inputs are identical bytes on both sides, so top-1 must match everywhere (ties included),
confidences within fp32-vs-fp64 rounding, and decisions / state bit-exactly except where a
confidence sits within that rounding of the threshold or of the transfer cut (counted).
"""
import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import decode
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import CONF_RTOL, bf16_to_f32, comparable_gate, comparable_transfer

pytestmark = pytest.mark.gpu


def _oracle(w, k, delta_p, m_req, gate_on, row_begin, scope="block", eos_id=None):
    """k < 0 -> schedule; row_begin < 0 -> rows follow the active block."""
    st = {n: np.array(v, dtype=np.int64) for n, v in w.state.items()}
    B = w.logits_bits.shape[0]
    n_blocks = (st["tokens"].shape[1] - w.prompt_len) // w.block_len
    outs = []
    for b in range(B):
        x = bf16_to_f32(w.logits_bits[b])
        outs.append(decode.step_row(st, b, x, w.prompt_len, w.block_len, w.steps_per_block,
                                    n_blocks, w.mask_id, delta_p, m_req, gate_on,
                                    k_override=None if k < 0 else k,
                                    logits_row0=None if row_begin < 0 else row_begin,
                                    scope=scope, eos_id=eos_id))
    return st, outs


def _gpu(w, k, delta_p, m_req, gate_on, row_begin, scope="block", eos_id=None):
    from paper_2608_11235_amd import DecodeState, Gate, Sched, vocab_gate
    B, R, V = w.logits_bits.shape
    L = w.state["tokens"].shape[1]
    st = DecodeState.from_host(w.state, w.prompt_len, L - w.prompt_len, R, w.block_len)
    logits = to_dev(w.logits_bits.view(np.int16))
    vocab_gate(logits, R, row_begin, V, w.mask_id, st, k,
               Sched(w.block_len, w.steps_per_block, eos_id),
               Gate(delta_p, m_req, gate_on, 1 if scope == "global" else 0))
    torch.cuda.synchronize()
    return st.to_host()


def _compare(w, gpu, st_or, outs, k, delta_p, gate_on, row_begin):
    B = w.logits_bits.shape[0]
    L = w.state["tokens"].shape[1]
    x_hat = np.stack([o["x_hat"] for o in outs])
    c = np.stack([o["c"] for o in outs])
    assert (gpu["top1"] == x_hat).all(), f"top-1 mismatches: {(gpu['top1'] != x_hat).sum()}"
    np.testing.assert_allclose(gpu["conf"], c, rtol=CONF_RTOL, atol=0)
    sched = decode.transfer_schedule(w.block_len, w.steps_per_block)
    excluded = 0
    for b in range(B):
        o = outs[b]
        lo = w.prompt_len + o["block"] * w.block_len
        pos = np.arange(lo, lo + w.block_len)
        row0 = row_begin if row_begin >= 0 else lo
        c_pos = np.zeros(L)
        c_pos[pos] = c[b, pos - row0]
        U_blk = pos[w.state["unresolved"][b, pos] == 1]
        kk = k if k >= 0 else int(sched[int(w.state["step_idx"][b])])
        ok = comparable_transfer(c_pos, U_blk, kk, 0.0)
        if gate_on:
            resid = np.setdiff1d(U_blk, o["T"])
            ok = ok and bool(np.all(comparable_gate(c_pos[resid], delta_p, 0.0)))
        if not ok:
            excluded += 1
            continue
        dec = np.zeros(w.block_len, np.int64)
        dec[o["T"] - lo] = 1
        dec[o["A"] - lo] = 2
        rem = np.asarray(o.get("removed", []), np.int64)
        dec[rem[(rem >= lo) & (rem < lo + w.block_len)] - lo] = 3
        assert (gpu["decision"][b] == dec).all(), f"batch row {b} decisions"
        for n in ("tokens", "unresolved", "prev_top1", "persist"):
            assert (gpu[n][b] == st_or[n][b]).all(), f"batch row {b} {n}"
        for n in ("block_idx", "step_idx"):
            assert gpu[n][b] == st_or[n][b], f"batch row {b} {n}"
        assert gpu["done"][b] == int(o["done"])
    print(f"excluded batch rows: {excluded}/{B}")
    return excluded


def _check(w, k, delta_p, m_req, gate_on, row_begin=0, scope="block", eos_id=None):
    gpu = _gpu(w, k, delta_p, m_req, gate_on, row_begin, scope, eos_id)
    st_or, outs = _oracle(w, k, delta_p, m_req, gate_on, row_begin, scope, eos_id)
    return _compare(w, gpu, st_or, outs, k, delta_p, gate_on, row_begin), gpu


CASES = [(0.65, 1, True), (0.05, 1, True), (0.2, 0, True), (0.5, 2, True), (0.65, 1, False)]


@pytest.mark.parametrize("delta_p,m_req,gate_on", CASES)
def test_vocab_gate_small(delta_p, m_req, gate_on):
    require_gpu()
    log_case(f"vocab_gate small dp={delta_p} m={m_req} gate={gate_on}")
    w = si.vocab_gate_workload(seed=2, batch=6, prompt_len=64, gen_len=128, vocab=5000,
                               mask_id=4990, block_len=32, steps_per_block=32,
                               masked_in_block=8, spike_max=12.0)
    ex, _ = _check(w, 1, delta_p, m_req, gate_on)
    assert ex <= 1


@pytest.mark.parametrize("step0", [False, True])
@pytest.mark.parametrize("delta_p,m_req,gate_on", [(0.65, 1, True), (0.2, 0, True), (0.0, 1, True),
                                                   (0.5, 2, True)])
def test_vocab_gate_global_scope(delta_p, m_req, gate_on, step0):
    """GLOBAL persistence scope (R5): counters of every scored unresolved position move,
    inside and outside the active block, and block step 0 does not reset them.  Includes
    the persistence-only variant (delta_p = 0, m = 1)."""
    require_gpu()
    log_case(f"vocab_gate global dp={delta_p} m={m_req} step0={step0}")
    w = si.vocab_gate_workload(seed=4, batch=5, prompt_len=32, gen_len=128, vocab=3001,
                               mask_id=17, block_len=32, steps_per_block=8,
                               masked_in_block=12, spike_max=11.0)
    if step0:
        w.state["step_idx"][:] = 0
    ex, gpu = _check(w, -1, delta_p, m_req, gate_on, 0, "global")
    assert ex <= 1
    # positions of later blocks were updated (BLOCK would leave them untouched)
    moved = 0
    for b in range(5):
        hi = 32 + 32 * (int(w.state["block_idx"][b]) + 1)
        later = np.arange(hi, w.state["tokens"].shape[1])
        later = later[w.state["unresolved"][b, later] == 1]
        moved += int((gpu["prev_top1"][b, later] != w.state["prev_top1"][b, later]).sum())
    assert moved > 0


@pytest.mark.parametrize("scope", ["block", "global"])
def test_vocab_gate_eos_aware(scope):
    """EOS-aware controller (R27): the EOS id is the top-1 of the highest-confidence
    unresolved position of batch row 0's block, so the transfer rule commits it there; the
    cut resolves every later unresolved position as EOS (decision 3 inside the block) and
    the row stops once its block is done.  Every state array must equal the oracle's."""
    require_gpu()
    log_case(f"vocab_gate eos-aware scope={scope}")
    w = si.vocab_gate_workload(seed=8, batch=4, prompt_len=16, gen_len=96, vocab=2000,
                               mask_id=1999, block_len=32, steps_per_block=4,
                               masked_in_block=20, spike_max=12.0)
    st0, outs0 = _oracle(w, 2, 0.5, 1, True, 0, scope)
    b0 = outs0[0]
    lo = 16 + 32 * int(w.state["block_idx"][0])
    T0 = np.asarray(b0["T"], np.int64)
    c_blk = b0["c"][T0]                       # rows start at canvas position 0
    eos = int(b0["x_hat"][T0[np.argmax(c_blk)]])
    ex, gpu = _check(w, 2, 0.5, 1, True, 0, scope, eos)
    assert ex <= 1
    st_or, outs = _oracle(w, 2, 0.5, 1, True, 0, scope, eos)
    cut = outs[0]["eos_cut"]
    assert cut is not None
    assert not gpu["unresolved"][0, cut + 1:].any()
    assert gpu["tokens"][0, cut] == eos


@pytest.mark.parametrize("V", [13, 2047, 2048])
def test_vocab_gate_odd_vocab_and_k(V):
    require_gpu()
    log_case(f"vocab_gate V={V}")
    w = si.vocab_gate_workload(seed=5, batch=3, prompt_len=8, gen_len=64, vocab=V, mask_id=V // 2,
                               block_len=16, steps_per_block=4, masked_in_block=10, spike_max=8.0)
    for k in (0, 3, 16, -1):
        ex, _ = _check(w, k, 0.3, 1, True)
        assert ex <= 1


def test_vocab_gate_ties_lowest_id():
    """Exact bf16 ties for the maximum resolve to the lowest token id; the mask id is skipped."""
    require_gpu()
    w = si.vocab_gate_workload(seed=7, batch=2, prompt_len=4, gen_len=32, vocab=1024, mask_id=3,
                               block_len=32, steps_per_block=8, masked_in_block=32, spike_max=0.0)
    bits = np.full_like(w.logits_bits, 0x3F80)   # every logit 1.0
    bits[:, :, 700] = 0x4000                     # 2.0 at 700 and 900: a tie
    bits[:, :, 900] = 0x4000
    bits[:, ::2, 3] = 0x4100                     # the mask id is larger on even rows
    w.logits_bits = bits
    gpu = _gpu(w, 2, 0.9, 0, True, 0)
    assert (gpu["top1"] == 700).all()
    np.testing.assert_allclose(gpu["conf"], np.e / (2 * np.e + 1021), rtol=CONF_RTOL)


def test_vocab_gate_block_rows_and_determinism():
    """Rows that follow each batch row's active block (row_begin < 0), schedule k, and
    bitwise repeatability of two identical calls."""
    require_gpu()
    w = si.vocab_gate_workload(seed=3, batch=4, prompt_len=16, gen_len=96, vocab=3000,
                               mask_id=2999, block_len=32, steps_per_block=8,
                               masked_in_block=20, spike_max=10.0)
    blk_bits = np.stack([w.logits_bits[b, 16 + 32 * int(w.state["block_idx"][b]):][:32]
                         for b in range(4)])
    wb = si.VocabGateWorkload(blk_bits, None, w.state, w.prompt_len, w.block_len,
                              w.steps_per_block, w.vocab, w.mask_id)
    g1 = _gpu(wb, -1, 0.4, 1, True, -1)
    g2 = _gpu(wb, -1, 0.4, 1, True, -1)
    for n in g1:
        assert (g1[n] == g2[n]).all(), n
    st_or, outs = _oracle(wb, -1, 0.4, 1, True, -1)
    assert _compare(wb, g1, st_or, outs, -1, 0.4, True, -1) <= 1


def test_vocab_gate_step0_reset_and_finished_rows():
    """Block step 0 resets counters (persistence is per block); finished rows are untouched."""
    require_gpu()
    w = si.vocab_gate_workload(seed=11, batch=3, prompt_len=8, gen_len=64, vocab=512,
                               mask_id=511, block_len=32, steps_per_block=4, masked_in_block=32,
                               spike_max=9.0)
    w.state["step_idx"][:] = 0
    w.state["block_idx"][2] = 2                  # finished row (n_blocks == 2)
    gpu = _gpu(w, -1, 0.5, 0, True, 0)
    st_or, outs = _oracle(w, -1, 0.5, 0, True, 0)
    for b in range(2):
        lo = 8 + 32 * int(w.state["block_idx"][b])
        assert (gpu["persist"][b, lo:lo + 32] == 0).all()
        assert (gpu["prev_top1"][b, lo:lo + 32] == st_or["prev_top1"][b, lo:lo + 32]).all()
    assert gpu["done"][2] == 1 and (gpu["decision"][2] == 0).all()
    for n in ("tokens", "unresolved", "prev_top1", "persist"):
        assert (gpu[n][2] == w.state[n][2]).all()
    assert gpu["block_idx"][2] == 2


@pytest.mark.slow
def test_vocab_gate_full_size():
    """The vocab/gate workload at full size: bf16 logits [8, 512, 126464], k = 1."""
    require_gpu()
    log_case("vocab_gate full size [8,512,126464]")
    w = si.vocab_gate_workload(seed=2)
    ex, _ = _check(w, 1, 0.65, 1, True)
    assert ex <= 1
