"""Parity at the full LLaDA-8B / Dream-7B widths (slow: minutes of CPU oracle time).

The GPU runs the real shapes (d 4096 / 3584, 32 or 28 x 128 heads, FFN 12288 / 18944,
vocab 126464 / 152064, canvas 512 or 1280, batch 1 or 8); the fp64 oracle recomputes
sampled outputs: a reduced layer count, the active-block rows, sampled batch rows.  The
full 32-layer pass is checked by properties that hold at any size (dense recovery, no
mask left, bitwise repeatability).
"""
import os

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import decode
from oracle import forward as of
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import (CONF_RTOL, bf16_to_f32, comparable_gate, comparable_transfer,
                          logit_tolerance, margins)

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def _canvas(spec, B, P, G, seed=1):
    prompt = si.prompt_tokens(seed, B, P, spec.vocab, spec.mask_id)
    return prompt, si.initial_decode_state(prompt, G, spec.mask_id)


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
                err = np.abs(got[b].astype(np.float64) - ref)
                tol = logit_tolerance(ref)
                print(f"  batch row {b}: max err {err.max():.4g} (tol {tol:.4g}; "
                      f"{err.max() / np.abs(ref).max():.4f} of max|l|), "
                      f"rel rms {np.sqrt(np.mean(err ** 2) / np.mean(ref ** 2)):.3g}")
                assert err.max() <= tol
                x_or, _ = decode.top1_confidence(ref, spec.mask_id)
                D = err.max(axis=-1)
                p1 = margins(ref, spec.mask_id) > 2 * D
                x_gpu = np.argmax(np.where(np.arange(spec.vocab) == spec.mask_id, -np.inf,
                                           got[b].astype(np.float64)), axis=-1)
                assert (x_gpu[p1] == x_or[p1]).all()


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


def test_llada_width_teacher_forced_step():
    """Decisions of one denoising step at full width (2 layers), teacher-forced from the
    oracle's state: block 0 step 0 of a fresh canvas."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = si.LLADA_8B.with_layers(2)
    P, G, BLK, S = 256, 256, 32, 32
    prompt, st = _canvas(spec, 1, P, G)
    w = si.HostWeights(spec, 0)
    ref = of.forward_logits(w, spec, st["tokens"], np.arange(P, P + BLK))[0]
    st_or = {k: v.astype(np.int64) for k, v in st.items()}
    o = decode.step_row(st_or, 0, ref, P, BLK, S, G // BLK, spec.mask_id, 0.65, 1, True)
    with Model(spec, seed=0, max_batch=1, max_seq=P + G) as m:
        got = bf16_to_f32(m.forward_logits(to_dev(st["tokens"]), P, BLK).cpu().numpy())[0]
        D = np.abs(got.astype(np.float64) - ref).max(axis=-1)
        ds = DecodeState.from_host(st, P, G, BLK, BLK)
        m.denoise_step(ds, Sched(BLK, S), Gate(0.65, 1, True))
        gpu = ds.to_host()
    p1 = margins(ref, spec.mask_id) > 2 * D
    assert (gpu["top1"][0][p1] == o["x_hat"][p1]).all()
    dlnc = np.abs(np.log(gpu["conf"][0].astype(np.float64)) - np.log(o["c"]))
    assert (dlnc <= 2 * D + CONF_RTOL).all()
    pos = np.arange(P, P + BLK)
    c_pos = np.zeros(P + G)
    c_pos[pos] = o["c"]
    D_pos = np.zeros(P + G)
    D_pos[pos] = D
    if comparable_transfer(c_pos, pos, o["k"], D_pos) and p1[(o["T"] - P)].all():
        want = np.zeros(BLK, np.int64)
        want[o["T"] - P] = 1
        assert (gpu["decision"][0] == want).all()
        assert (gpu["tokens"][0][o["T"]] == o["x_hat"][o["T"] - P]).all()
    # random-init confidences (~1e-3) never reach 0.65 and m is 0 at block step 0: no gate
    assert (gpu["decision"][0] != 2).all()
    assert gpu["step_idx"][0] == 1 and gpu["block_idx"][0] == 0
    print(f"  max logit err {D.max():.4g}, top-1 comparable {p1.sum()}/32")


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


@pytest.mark.skipif(os.environ.get("CORA_FULL_DEPTH_ORACLE") == "0",
                    reason="CORA_FULL_DEPTH_ORACLE=0 skips the full 32-layer fp64 oracle pass")
def test_llada_full_depth_logits():
    require_gpu()
    _check_rows(si.LLADA_8B, 1, 256, 256, [(256, 32)], [0], 32)
