"""Step decisions against the oracle's rules on the GPU's own logits (tests/own_logits.py).

Every step of the GPU's own decode is checked: the oracle applies Eqs. (1)-(4), the transfer
rule and termination to the bf16 logits the GPU computes for the pre-step state, and the
step's top-1, confidence, decisions and written state must match wherever the fp32-vs-fp64
rounding of the confidence cannot flip a cut or a threshold (>= 95 % of decisions).

Configurations: the paper-shaped tiny model (2 layers, d 256, vocab 2048, logits x8) over
every step of both blocks, BLOCK and GLOBAL persistence scope, four gate settings and the
EOS-aware controller; the Dream-7B width (GQA 28/4, QKV bias, vocab 152064) at B = 8 with 2
layers; the LLaDA-8B width on the 1280-position canvas with 1 layer.
"""
from dataclasses import replace

import numpy as np
import pytest

import seeded_inputs as si
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.own_logits import run_decode

pytestmark = pytest.mark.gpu

P, G, BLK, S = 32, 64, 32, 16
GATES = [(0.65, 1, True), (0.3, 0, True), (0.65, 1, False), (0.1, 2, True)]
MIN_FRAC = 0.95


def _report(tag, compared, total, steps):
    frac = compared / max(total, 1)
    print(f"[summary] {tag}: steps {steps}, decisions compared {compared}/{total} ({frac:.3f})")
    assert steps > 0 and total > 0
    assert compared >= MIN_FRAC * total, f"{tag}: only {compared}/{total} compared"


@pytest.mark.parametrize("scope", ["block", "global"])
@pytest.mark.parametrize("delta_p,m_req,gate_on", GATES)
def test_tiny_own_logits(delta_p, m_req, gate_on, scope):
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = si.TINY
    B = 2
    prompt = si.prompt_tokens(1, B, P, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, G, spec.mask_id)
    sc = 0 if scope == "block" else 1
    tag = f"tiny {scope} dp={delta_p} m={m_req} gate={gate_on}"
    log_case(tag)
    with Model(spec, seed=0, max_batch=B, max_seq=P + G) as m:
        st = DecodeState.from_host(host, P, G, BLK if sc == 0 else G, BLK)
        c, t, n = run_decode(m, st, Sched(BLK, S), Gate(delta_p, m_req, gate_on, sc), spec, P,
                             G, scope)
    _report(tag, c, t, n)


@pytest.mark.parametrize("scope", ["block", "global"])
def test_tiny_own_logits_eos(scope):
    """EOS-aware controller (Table 2): the EOS id is a token the GPU's fixed-horizon decode
    commits early in block 0, so the cut happens and later positions are removed."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = si.TINY
    B = 2
    prompt = si.prompt_tokens(1, B, P, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, G, spec.mask_id)
    sc = 0 if scope == "block" else 1
    gate = Gate(0.3, 1, True, sc)
    with Model(spec, seed=0, max_batch=B, max_seq=P + G) as m:
        y, _, _ = m.block_decode(to_dev(prompt), G, Sched(BLK, S), gate)
        eos = int(y.cpu().numpy()[0, P + 6])
        tag = f"tiny eos={eos} {scope}"
        log_case(tag)
        st = DecodeState.from_host(host, P, G, BLK if sc == 0 else G, BLK)
        c, t, n = run_decode(m, st, Sched(BLK, S, eos), gate, spec, P, G, scope, eos_id=eos)
        fin = st.to_host()
    assert (fin["tokens"][:, P:] != spec.mask_id).all()
    assert (fin["tokens"][0, P:] == eos).sum() > 1, "the EOS cut should remove positions"
    _report(tag, c, t, n)


def test_dream_width_b8_own_logits():
    """Dream-7B width (GQA 28/4, QKV bias, theta 1e6, eps 1e-6, vocab 152064), 2 layers,
    batch 8, prompt 256 + gen 256: the first 6 steps of block 0."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = si.DREAM_7B.with_layers(2)
    B, Pd, Gd = 8, 256, 256
    prompt = si.prompt_tokens(1, B, Pd, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, Gd, spec.mask_id)
    log_case("dream7b-2L B=8 own logits")
    with Model(spec, seed=0, max_batch=B, max_seq=Pd + Gd) as m:
        st = DecodeState.from_host(host, Pd, Gd, 32, 32)
        c, t, n = run_decode(m, st, Sched(32, 32), Gate(0.65, 1, True), spec, Pd, Gd,
                             max_steps=6)
    _report("dream7b-2L B=8", c, t, n)


def test_llada_long_canvas_own_logits():
    """LLaDA-8B width on the 1280-position canvas (prompt 256 + gen 1024), 1 layer: the
    first 4 steps of block 0, gate on."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = si.LLADA_8B.with_layers(1)
    Pd, Gd = 256, 1024
    prompt = si.prompt_tokens(1, 1, Pd, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, Gd, spec.mask_id)
    log_case("llada8b-1L L=1280 own logits")
    with Model(spec, seed=0, max_batch=1, max_seq=Pd + Gd) as m:
        st = DecodeState.from_host(host, Pd, Gd, 32, 32)
        c, t, n = run_decode(m, st, Sched(32, 32), Gate(0.65, 1, True), spec, Pd, Gd,
                             max_steps=4)
    _report("llada8b-1L L=1280", c, t, n)


def test_llada_width_gated_x8_own_logits():
    """LLaDA-8B width, 2 layers, logits x8 (so confidences spread and the gate fires; not a
    paper configuration), batch 3: a whole 2-block decode with the gate on."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = replace(si.LLADA_8B.with_layers(2), logit_scale=8.0)
    B, Pd, Gd = 3, 256, 64
    prompt = si.prompt_tokens(2, B, Pd, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, Gd, spec.mask_id)
    log_case("llada8b-2L x8 B=3 own logits")
    with Model(spec, seed=0, max_batch=B, max_seq=Pd + Gd) as m:
        st = DecodeState.from_host(host, Pd, Gd, 32, 32)
        c, t, n = run_decode(m, st, Sched(32, 32), Gate(0.65, 1, True), spec, Pd, Gd)
        passes = st.to_host()["passes"]
    print(f"  passes per block {passes.tolist()}")
    _report("llada8b-2L x8 B=3", c, t, n)
