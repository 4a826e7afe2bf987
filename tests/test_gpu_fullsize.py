"""Parity at the full LLaDA-8B / Dream-7B widths (slow: minutes of CPU oracle time).

The GPU runs the real shapes (d 4096 / 3584, 32 or 28 x 128 heads, FFN 12288 / 18944,
vocab 126464 / 152064, canvas 512 or 1280, batch 1 or 8); the fp64 oracle recomputes
sampled outputs: a reduced layer count, the active-block rows, sampled batch rows, and two
seeded spot steps at the full 32 layers (logits, top-1, confidence, decisions, counters).
The full 32-layer decode is also checked by properties that hold at any size (dense
recovery, no mask left, bitwise repeatability).
"""
import os

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import decode
from oracle import forward as of
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import (FULL_DEPTH_RANGE_CASE, bf16_to_f32, comparable_decisions,
                          describe_error, logit_tolerance, margins, range_tolerance)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _canvas(spec, B, P, G, seed=1):
    prompt = si.prompt_tokens(seed, B, P, spec.vocab, spec.mask_id)
    return prompt, si.initial_decode_state(prompt, G, spec.mask_id)


def _check_logits(got_b, ref, tag, range_case=False):
    """max |l_gpu - l_oracle| within 2e-2 max|l| (range-scaled for the one marked case)."""
    err = np.abs(got_b.astype(np.float64) - ref)
    tol = range_tolerance(ref) if range_case else logit_tolerance(ref)
    kind = f"range bound: {FULL_DEPTH_RANGE_CASE}" if range_case else "max|l| bound"
    print(f"  {tag}: {describe_error(err.max(), ref)} (tol {tol:.4g}, {kind}), "
          f"rel rms {np.sqrt(np.mean(err ** 2) / np.mean(ref ** 2)):.3g}")
    assert err.max() <= tol
    return err.max(axis=-1)


def _check_rows(spec, B, P, G, row_sets, oracle_rows_b, n_layers):
    from paper_2608_11235_amd import Model
    spec = spec.with_layers(n_layers)
    prompt, st = _canvas(spec, B, P, G)
    L = P + G
    w = si.HostWeights(spec, 0)
    with Model(spec, seed=0, max_batch=B, max_seq=L) as m:
        for r0, n in row_sets:
            log_case(f"{spec.name} B={B} L={L} rows [{r0},{r0 + n})")
            got = bf16_to_f32(m.forward_logits(to_dev(st["tokens"]), r0, n).cpu().numpy())
            for b in oracle_rows_b:
                ref = of.forward_logits(w, spec, st["tokens"][b:b + 1], np.arange(r0, r0 + n))[0]
                D = _check_logits(got[b], ref, f"batch row {b}")
                x_or, _ = decode.top1_confidence(ref, spec.mask_id)
                p1 = margins(ref, spec.mask_id) > 2 * D
                x_gpu = np.argmax(np.where(np.arange(spec.vocab) == spec.mask_id, -np.inf,
                                           got[b].astype(np.float64)), axis=-1)
                assert (x_gpu[p1] == x_or[p1]).all()
                print(f"    top-1 compared {int(p1.sum())}/{n}")


def test_llada_width_two_layers():
    require_gpu()
    _check_rows(si.LLADA_8B, 1, 256, 256, [(256, 32), (0, 8)], [0], 2)


def test_llada_long_canvas_one_layer():
    """The 1280-position canvas (prompt 256 + 1024 generated)."""
    require_gpu()
    _check_rows(si.LLADA_8B, 1, 256, 1024, [(256, 32), (1248, 32)], [0], 1)


def test_dream_width_batch8_two_layers():
    """GQA 28/4, QKV bias, theta 1e6, eps 1e-6, batch 8; oracle on two sampled rows."""
    require_gpu()
    _check_rows(si.DREAM_7B, 8, 256, 256, [(256, 32)], [0, 5], 2)


def _spot_states(spec, P, G, w, blk=32):
    """Seeded pre-step states at the LLaDA-8B shape (B = 1), with the oracle logits of their
    active block: the fresh canvas (block 0, step 0), and a mid-decode state (block 4, step 5:
    blocks 0-3 and 5 positions of block 4 committed with seeded tokens; previous top-1 of the
    other block-4 positions set to the oracle's top-1 for half of them, seeded otherwise, and
    counters drawn from {0..3}, so the persistence update and the gate see real histories)."""
    rng = np.random.default_rng(11)
    prompt, st0 = _canvas(spec, 1, P, G)
    lo0 = P
    yield "block 0 step 0", st0, lo0, of.forward_logits(w, spec, st0["tokens"],
                                                        np.arange(lo0, lo0 + blk))[0]
    st = {k: v.copy() for k, v in st0.items()}
    lo = P + 4 * blk
    done = np.arange(P, lo).tolist() + (lo + rng.choice(blk, 5, replace=False)).tolist()
    vocab_ids = np.delete(np.arange(spec.vocab), spec.mask_id)
    st["tokens"][0, done] = rng.choice(vocab_ids, len(done))
    st["unresolved"][0, done] = 0
    st["block_idx"][0], st["step_idx"][0] = 4, 5
    ref = of.forward_logits(w, spec, st["tokens"], np.arange(lo, lo + blk))[0]
    x_or, _ = decode.top1_confidence(ref, spec.mask_id)
    open_ = np.nonzero(st["unresolved"][0, lo:lo + blk])[0]
    half = rng.random(len(open_)) < 0.5
    st["prev_top1"][0, lo + open_] = np.where(half, x_or[open_], rng.choice(vocab_ids, len(open_)))
    st["persist"][0, lo + open_] = rng.integers(0, 4, len(open_))
    yield "block 4 step 5", st, lo, ref


def _teacher_forced_spot_steps(n_layers, range_case):
    """Decisions of one denoising step at full width, teacher-forced from seeded states:
    against the fp64 oracle where the measured logit error cannot flip them (P1-P3), and
    against the oracle's rules on the GPU's own logits (tests/own_logits.py)."""
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    from tests.own_logits import check_step
    spec = si.LLADA_8B.with_layers(n_layers)
    P, G, BLK, S = 256, 256, 32, 32
    w = si.HostWeights(spec, 0)
    for i in range(n_layers):                       # seeded host weights, with progress
        w.layer(i)
        if i % 8 == 7:
            print(f"    host weights: layer {i + 1} of {n_layers}", flush=True)
    gate = Gate(0.65, 1, True)
    tot = {"top1": 0, "dec": 0, "rows": 0, "U": 0, "own": 0, "own_U": 0}
    with Model(spec, seed=0, max_batch=1, max_seq=P + G) as m:
        for tag, st, lo, ref in _spot_states(spec, P, G, w, BLK):
            log_case(f"{spec.name} teacher-forced {tag}")
            st_or = {k: v.astype(np.int64) for k, v in st.items()}
            o = decode.step_row(st_or, 0, ref, P, BLK, S, G // BLK, spec.mask_id, gate.delta_p,
                                gate.m_req, True)
            got = bf16_to_f32(m.forward_logits(to_dev(st["tokens"]), lo, BLK).cpu().numpy())[0]
            D = _check_logits(got, ref, tag, range_case)
            ds = DecodeState.from_host(st, P, G, BLK, BLK)
            m.denoise_step(ds, Sched(BLK, S), gate)
            gpu = ds.to_host()
            U = st["unresolved"][0][lo:lo + BLK] == 1
            gam = margins(ref, spec.mask_id)
            dec_ok, p1 = comparable_decisions(o["c"], gam, np.asarray(o["T"]) - lo, o["k"], U,
                                              D, gate.delta_p, True)
            # Eq. (1): top-1 where the margin survives the error, confidence within 2 D
            assert (gpu["top1"][0][p1] == o["x_hat"][p1]).all(), f"{tag}: top-1"
            dlnc = np.abs(np.log(gpu["conf"][0].astype(np.float64)) - np.log(o["c"]))
            assert (dlnc <= 2 * D + 1e-4).all(), f"{tag}: confidence"
            want = np.zeros(BLK, np.int64)
            want[np.asarray(o["T"], np.int64) - lo] = 1
            want[np.asarray(o["A"], np.int64) - lo] = 2
            cmp = dec_ok & U
            assert (gpu["decision"][0][cmp] == want[cmp]).all(), f"{tag}: decisions"
            # counters (Eq. 2) of positions with a certain top-1
            sel = U & p1
            for n in ("prev_top1", "persist"):
                assert (gpu[n][0][lo:lo + BLK][sel] == st_or[n][0][lo:lo + BLK][sel]).all(), \
                    f"{tag}: {n}"
            tot["top1"] += int(p1.sum())
            tot["rows"] += BLK
            tot["dec"] += int(cmp.sum())
            tot["U"] += int(U.sum())
            print(f"    {tag}: top-1 compared {int(p1.sum())}/{BLK}, decisions compared "
                  f"{int(cmp.sum())}/{int(U.sum())}, transfer T oracle {o['T'].tolist()} "
                  f"gpu {(np.nonzero(gpu['decision'][0] == 1)[0] + lo).tolist()}")
            # the same step on the GPU's own logits: every decision outside fp32 rounding
            ds = DecodeState.from_host(st, P, G, BLK, BLK)
            c, t = check_step(m, ds, Sched(BLK, S), gate, spec, P, G)
            tot["own"] += c
            tot["own_U"] += t
    print(f"[summary] {spec.name}: fp64 oracle: top-1 {tot['top1']}/{tot['rows']}, decisions "
          f"{tot['dec']}/{tot['U']}; own logits: decisions {tot['own']}/{tot['own_U']}")
    assert tot["top1"] > 0 and tot["dec"] > 0
    assert tot["own"] >= 0.95 * tot["own_U"]


def test_llada_width_teacher_forced_step():
    """2 layers at the LLaDA-8B width: logits within the max|l| bound and step decisions."""
    require_gpu()
    _teacher_forced_spot_steps(2, range_case=False)


@pytest.mark.skipif(os.environ.get("CORA_FULL_DEPTH_ORACLE") == "0",
                    reason="CORA_FULL_DEPTH_ORACLE=0 skips the full 32-layer fp64 oracle passes")
def test_llada_full_depth_teacher_forced_step():
    """All 32 layers at L = 512: the one case held to the range-scaled logit bound
    (FULL_DEPTH_RANGE_CASE, tests/parity.py), with top-1, confidence, transfer and gate
    decisions and counters compared against the fp64 oracle (P1-P3) and every decision
    compared on the GPU's own logits."""
    require_gpu()
    _teacher_forced_spot_steps(32, range_case=True)


def test_llada_full_depth_decode_properties():
    """All 32 layers, gen 256: dense recovery, no mask left, bitwise repeatable decode."""
    require_gpu()
    from paper_2608_11235_amd import Gate, Model, Sched
    spec = si.LLADA_8B
    P, G = 256, 256
    prompt, _ = _canvas(spec, 1, P, G)
    with Model(spec, seed=0, max_batch=1, max_seq=P + G) as m:
        log_case("llada8b full depth block decode (gate off, then on twice)")
        out0, passes0, total0 = m.block_decode(to_dev(prompt), G, Sched(32, 32), Gate(0.65, 1, False))
        assert (passes0 == 32).all() and total0 == 256
        out1, passes1, _ = m.block_decode(to_dev(prompt), G, Sched(32, 32), Gate(0.65, 1, True))
        out2, passes2, _ = m.block_decode(to_dev(prompt), G, Sched(32, 32), Gate(0.65, 1, True))
        out0, out1, out2 = out0.cpu().numpy(), out1.cpu().numpy(), out2.cpu().numpy()
    assert (out1 == out2).all() and (passes1 == passes2).all()
    assert (out1[:, P:] != spec.mask_id).all() and (out1[:, :P] == prompt).all()
    # the gate is inert at random init: same passes and tokens as dense recovery
    assert (passes1 == 32).all() and (out1 == out0).all()
