"""cora_vocab_gate_noalloc (the vocab/gate kernels with a fixed scratch array, for callers
that cannot allocate) through the C ABI, against cora_vocab_gate on the same inputs.

Three calls in a row, each smaller than the one before: 4 x 512 rows of the 126464-entry
vocabulary (one part per row), then 32 block-following rows of one batch row (the row split
over 15 workgroups), then an odd 50001-entry vocabulary (no 16-byte chunks, 6 parts per
row).  The same inputs go through both entry points: top-1 must agree bit for bit, the
confidence within fp32 summation-order rounding, and decisions and state bit for bit except
in a batch row whose transfer cut or gate threshold lies within that rounding (at most one
such row, and it is counted)."""
import numpy as np
import pytest
import torch

import seeded_inputs as si
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import comparable_decisions
from oracle import decode

pytestmark = pytest.mark.gpu

RTOL = 2e-5
STATE = ("tokens", "unresolved", "prev_top1", "persist", "block_idx", "step_idx", "done")


def _run(fn, w, logits_bits, row_begin, k, gate):
    from paper_2608_11235_amd import DecodeState, Sched
    B, R, V = logits_bits.shape
    L = w.state["tokens"].shape[1]
    st = DecodeState.from_host(w.state, w.prompt_len, L - w.prompt_len, R, w.block_len)
    logits = to_dev(np.ascontiguousarray(logits_bits).view(np.int16))
    fn(logits, R, row_begin, V, w.mask_id, st, k, Sched(w.block_len, w.steps_per_block), gate)
    torch.cuda.synchronize()
    return st.to_host()


def _case(w, logits_bits, row_begin, k, gate):
    from paper_2608_11235_amd import vocab_gate, vocab_gate_noalloc
    ref = _run(vocab_gate, w, logits_bits, row_begin, k, gate)
    got = _run(vocab_gate_noalloc, w, logits_bits, row_begin, k, gate)
    assert (got["top1"] == ref["top1"]).all(), f"top-1: {(got['top1'] != ref['top1']).sum()} differ"
    rel = np.abs(got["conf"].astype(np.float64) / ref["conf"].astype(np.float64) - 1.0)
    assert rel.max() <= RTOL, f"confidence rel diff {rel.max():.3g}"
    B = logits_bits.shape[0]
    uncertain = 0
    sched = decode.transfer_schedule(w.block_len, w.steps_per_block)
    for b in range(B):
        same = (got["decision"][b] == ref["decision"][b]).all() and \
            all((np.asarray(got[n][b]) == np.asarray(ref[n][b])).all() for n in STATE)
        if same:
            continue
        # only a decision within the two confidences' rounding may differ
        blk = int(w.state["block_idx"][b])
        lo = w.prompt_len + blk * w.block_len
        off = lo - row_begin if row_begin >= 0 else 0
        c = ref["conf"][b][off:off + w.block_len].astype(np.float64)
        U = w.state["unresolved"][b][lo:lo + w.block_len] == 1
        kk = k if k >= 0 else int(sched[int(w.state["step_idx"][b])])
        T = np.nonzero(ref["decision"][b] == 1)[0]
        ok, _ = comparable_decisions(c, np.full(len(c), np.inf), T, kk, U, 0.0, gate.delta_p,
                                     gate.enabled, 2 * RTOL)
        assert not ok[U].all(), f"batch row {b}: decisions differ where the cut is certain"
        uncertain += 1
    assert uncertain <= 1, f"{uncertain} batch rows differ"
    return uncertain


def test_noalloc_matches_vocab_gate():
    require_gpu()
    from paper_2608_11235_amd import Gate
    gate = Gate(0.65, 1, True)
    # 1: 4 x 512 rows (the whole canvas), vocab 126464
    log_case("noalloc call 1: B=4 x 512 rows, V=126464, fixed rows")
    w = si.vocab_gate_workload(seed=2, batch=4)
    u1 = _case(w, w.logits_bits, 0, 1, gate)
    # 2: smaller: one batch row, its 32 active-block rows, the schedule's k
    log_case("noalloc call 2: B=1 x 32 block rows, V=126464")
    w = si.vocab_gate_workload(seed=9, batch=1)
    lo = w.prompt_len + int(w.state["block_idx"][0]) * w.block_len
    u2 = _case(w, w.logits_bits[:, lo:lo + w.block_len], -1, -1, Gate(0.05, 1, True))
    # 3: smaller still: odd vocabulary (element loop), 2 x 32 block rows
    log_case("noalloc call 3: B=2 x 32 block rows, V=50001")
    w = si.vocab_gate_workload(seed=5, batch=2, prompt_len=16, gen_len=64, vocab=50001,
                               mask_id=25000)
    bits = np.stack([w.logits_bits[b, w.prompt_len + int(w.state["block_idx"][b]) * 32:][:32]
                     for b in range(2)])
    u3 = _case(w, bits, -1, -1, Gate(0.2, 0, True))
    print(f"[summary] rows within rounding: {u1}, {u2}, {u3}")


def test_noalloc_rejects_rows_beyond_scratch():
    """More rows than the fixed scratch holds: CORA_ERR_UNSUPPORTED, nothing launched, and
    the entry point works normally afterwards."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Sched, vocab_gate_noalloc
    from paper_2608_11235_amd._lib import CoraError
    B, P, G, V = 520, 0, 512, 8
    st = DecodeState(B, P, G, G, 32)
    logits = torch.zeros((B, G, V), dtype=torch.int16, device="cuda")
    with pytest.raises(CoraError) as e:
        vocab_gate_noalloc(logits, G, 0, V, 7, st, 1, Sched(32, 32), Gate(0.65, 1, True))
    assert e.value.status == -2 and "fixed scratch" in str(e.value)
    w = si.vocab_gate_workload(seed=3, batch=2, prompt_len=16, gen_len=64, vocab=4096,
                               mask_id=11)
    _case(w, w.logits_bits, 0, 1, Gate(0.65, 1, True))
