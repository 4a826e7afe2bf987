"""GPU parity of the whole denoising step and of the gated block decode (tiny config).

Teacher forcing: the oracle decodes with its fp64 forward and records the state before
every executed pass; the GPU step starts from that exact state.  Its block-row logits must
lie within the logit tolerance, and every decision that the measured logit error cannot
flip (P1-P3 in tests/parity.py) must match bit-exactly, along with the state it writes.

Free running: the GPU and the oracle each decode from the same prompt on their own.  They
must agree step for step until the first step holding a decision the logit error could
flip; after it the trajectories may legitimately differ.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import decode
from oracle import forward as of
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import (CONF_RTOL, bf16_to_f32, comparable_decisions, describe_error,
                          logit_tolerance, margins)

pytestmark = pytest.mark.gpu

SPEC = si.TINY
# With N(0, 0.02) weights every masked position sees the same input and near-uniform
# attention, so block confidences differ by ~1e-3 in ln c: almost every transfer cut is
# within the bf16 logit error and excluded.  The same shape drawn with std 0.07 (logits x2)
# spreads confidences and margins while bf16 activation rounding stays under 1.4 % of the
# largest logit, so over half of the decisions are comparable; it is an extra parity model.
# On the tiny model itself only a few decisions per decode clear the bf16 error (3/488 and
# 4/544 measured), so there the test requires a nonzero count; the step's decision logic at
# that config is compared on nearly every position against the oracle run on the GPU's own
# logits (tests/test_gpu_own_logits.py).
SEPARATED = replace(si.TINY, name="tiny-std0.07", init_std=0.07, logit_scale=2.0)
MODELS = [pytest.param(SPEC, 0.0, id="tiny"), pytest.param(SEPARATED, 0.4, id="tiny-std0.07")]
P, G, BLK, S = 32, 64, 32, 16
L = P + G


def _logits_fn(spec=SPEC):
    w = si.HostWeights(spec, 0)

    def fn(tokens, rows):
        return list(of.forward_logits(w, spec, tokens, rows))
    return fn


def _comparable(o, pre_unres, lo, D, delta_p, gate_on, blk=BLK):
    """Decision and top-1 comparability of the block positions (P1-P3, tests/parity.py)."""
    U = pre_unres[lo:lo + blk] == 1
    return comparable_decisions(o["c"], o["gamma"], np.asarray(o["T"]) - lo, o["k"], U, D,
                                delta_p, gate_on)


@pytest.mark.parametrize("spec,min_frac", MODELS)
@pytest.mark.parametrize("delta_p,m_req,gate_on", [(0.65, 1, True), (0.3, 0, True),
                                                   (0.65, 1, False), (0.1, 1, True)])
def test_teacher_forced_steps(delta_p, m_req, gate_on, spec, min_frac):
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    prompt = si.prompt_tokens(1, 1, P, spec.vocab, spec.mask_id)
    _, _, trace = decode.block_decode(_logits_fn(spec), prompt, G, spec.mask_id, BLK, S, delta_p,
                                      m_req, gate_on, record=True)
    n_dec = n_dec_ok = 0
    worst, worst_desc = 0.0, ""
    with Model(spec, seed=0, max_batch=1, max_seq=L) as m:
        for si_, step in enumerate(trace):
            log_case(f"teacher-forced {spec.name} step {si_} dp={delta_p} m={m_req} gate={gate_on}")
            pre, o = step["pre"], step["out"][0]
            lo = P + o["block"] * BLK
            lg = bf16_to_f32(m.forward_logits(to_dev(pre["tokens"].astype(np.int32)), lo, BLK)
                             .cpu().numpy())[0].astype(np.float64)
            ref = step["logits"][0]
            D = np.max(np.abs(lg - ref), axis=-1)
            if D.max() / np.max(np.abs(ref)) > worst:
                worst, worst_desc = D.max() / np.max(np.abs(ref)), describe_error(D.max(), ref)
            assert D.max() <= logit_tolerance(ref), f"step {si_}: {describe_error(D.max(), ref)}"
            st = DecodeState.from_host(pre, P, G, BLK, BLK)
            m.denoise_step(st, Sched(BLK, S), Gate(delta_p, m_req, gate_on))
            gpu = st.to_host()
            o = dict(o, gamma=margins(ref, spec.mask_id))
            dec_ok, p1 = _comparable(o, pre["unresolved"][0], lo, D, delta_p, gate_on)
            # Eq. (1): top-1 where the margin survives, confidence within the error bound
            assert (gpu["top1"][0][p1] == o["x_hat"][p1]).all(), f"step {si_} top-1"
            dlnc = np.abs(np.log(gpu["conf"][0].astype(np.float64)) - np.log(o["c"]))
            assert (dlnc <= 2 * D + CONF_RTOL).all(), f"step {si_} confidence"
            want = np.zeros(BLK, np.int64)
            want[np.asarray(o["T"], np.int64) - lo] = 1
            want[np.asarray(o["A"], np.int64) - lo] = 2
            assert (gpu["decision"][0][dec_ok] == want[dec_ok]).all(), f"step {si_} decisions"
            U = pre["unresolved"][0][lo:lo + BLK] == 1
            n_dec += int(U.sum())
            n_dec_ok += int((dec_ok & U).sum())
            # state written by the step: outside the block it must be untouched
            nxt = trace[si_ + 1]["pre"] if si_ + 1 < len(trace) else None
            if nxt is None:
                continue
            outside = np.ones(L, bool)
            outside[lo:lo + BLK] = False
            for n in ("tokens", "unresolved", "prev_top1", "persist"):
                assert (gpu[n][0][outside] == pre[n][0][outside]).all(), f"step {si_} {n}"
            blk = slice(lo, lo + BLK)
            same = dec_ok & (p1 | (want == 0))
            for n in ("unresolved", "tokens"):
                assert (gpu[n][0][blk][same] == nxt[n][0][blk][same]).all(), f"step {si_} {n}"
            for n in ("prev_top1", "persist"):
                assert (gpu[n][0][blk][p1] == nxt[n][0][blk][p1]).all(), f"step {si_} {n}"
            if dec_ok.all():
                for n in ("block_idx", "step_idx"):
                    assert (gpu[n] == nxt[n]).all(), f"step {si_} {n}"
    print(f"[summary] steps {len(trace)}: unresolved-position decisions compared "
          f"{n_dec_ok}/{n_dec}, worst step: {worst_desc}")
    assert n_dec_ok >= max(min_frac * n_dec, 1)


@pytest.mark.parametrize("spec,min_frac", MODELS)
@pytest.mark.parametrize("blk,steps", [(32, 16), (4, 4)])
@pytest.mark.parametrize("delta_p,m_req,gate_on", [(0.65, 1, True), (0.3, 0, True),
                                                   (0.65, 1, False), (0.0, 0, True)])
def test_free_running_decode(delta_p, m_req, gate_on, blk, steps, spec, min_frac):
    """GPU steps vs oracle steps from the same prompt, each on its own trajectory; and the
    block_decode entry point equal to the GPU's own step-by-step trajectory."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    log_case(f"free-running tiny dp={delta_p} m={m_req} gate={gate_on}")
    prompt = si.prompt_tokens(1, 2, P, spec.vocab, spec.mask_id)
    fn = _logits_fn(spec)
    host = si.initial_decode_state(prompt, G, spec.mask_id)
    st_or = {k: v.astype(np.int64) for k, v in host.items()}
    n_blocks = G // blk
    diverged = [None, None]
    agreed_steps = 0
    with Model(spec, seed=0, max_batch=2, max_seq=L) as m:
        st = DecodeState.from_host(host, P, G, blk, blk)
        sched, gate = Sched(blk, steps), Gate(delta_p, m_req, gate_on)
        for step in range(n_blocks * steps):
            gpu_pre = st.to_host()
            if (gpu_pre["block_idx"] >= n_blocks).all():
                break
            m.denoise_step(st, sched, gate)
            gpu = st.to_host()
            rows = [decode.block_positions(st_or, b, P, blk, n_blocks) for b in range(2)]
            logits = fn(st_or["tokens"].copy(), rows)
            for b in range(2):
                if diverged[b] is not None or st_or["block_idx"][b] >= n_blocks:
                    continue
                lo = rows[b][0]
                pre_unres = st_or["unresolved"][b].copy()
                o = decode.step_row(st_or, b, logits[b], P, blk, steps, n_blocks, spec.mask_id,
                                    delta_p, m_req, gate_on)
                o = dict(o, gamma=margins(logits[b], spec.mask_id))
                # before divergence both sides hold the same canvas: measure the error there
                lg = bf16_to_f32(m.forward_logits(to_dev(gpu_pre["tokens"][b:b + 1]), lo, blk)
                                 .cpu().numpy())[0].astype(np.float64)
                D = np.max(np.abs(lg - logits[b]), axis=-1)
                assert D.max() <= logit_tolerance(logits[b])
                dec_ok, p1 = _comparable(o, pre_unres, lo, D, delta_p, gate_on, blk)
                same = all((gpu[n][b] == st_or[n][b]).all() for n in
                           ("tokens", "unresolved", "block_idx", "step_idx"))
                if not same:
                    assert not (dec_ok.all() and p1[pre_unres[lo:lo + blk] == 1].all()), \
                        f"row {b} step {step}: diverged on a comparable step"
                    diverged[b] = step
            agreed_steps += 1
        final = st.to_host()
        out, passes, total = m.block_decode(to_dev(prompt), G, sched, gate)
        assert (out.cpu().numpy() == final["tokens"]).all(), "block_decode != step-by-step"
        assert (passes == final["passes"]).all()
    if not gate_on:
        assert (passes == steps).all() and total == n_blocks * steps
    if delta_p <= 0 and m_req == 0:
        assert (passes == 1).all()
    if gate_on and m_req >= 1:
        assert (passes >= 2).all()
    assert (final["tokens"][:, P:] != spec.mask_id).all()
    print(f"[summary] steps run {agreed_steps}, first divergence per row {diverged}, "
          f"passes {passes.tolist()}")


@pytest.mark.parametrize("spec,min_frac", MODELS)
@pytest.mark.parametrize("delta_p,m_req,gate_on", [(0.65, 1, True), (0.3, 0, True),
                                                   (0.0, 1, True), (0.1, 2, True)])
def test_global_scope_teacher_forced_steps(delta_p, m_req, gate_on, spec, min_frac):
    """GLOBAL persistence scope (R5): the step scores the whole generation region (LM head
    and row reduction in chunks), moves every scored unresolved counter, and gates the
    active block.  Teacher-forced from the oracle's global-scope trajectory."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    prompt = si.prompt_tokens(1, 1, P, spec.vocab, spec.mask_id)
    _, _, trace = decode.block_decode(_logits_fn(spec), prompt, G, spec.mask_id, BLK, S, delta_p,
                                      m_req, gate_on, record=True, scope="global")
    n_dec = n_dec_ok = 0
    gen = slice(P, L)
    with Model(spec, seed=0, max_batch=1, max_seq=L) as m:
        for si_, step in enumerate(trace):
            log_case(f"global teacher-forced {spec.name} step {si_} dp={delta_p} m={m_req}")
            pre, o = step["pre"], step["out"][0]
            lo = P + o["block"] * BLK
            ref = step["logits"][0]                                   # rows P .. L-1
            lg = bf16_to_f32(m.forward_logits(to_dev(pre["tokens"].astype(np.int32)), P, G)
                             .cpu().numpy())[0].astype(np.float64)
            Dall = np.max(np.abs(lg - ref), axis=-1)
            assert Dall.max() <= logit_tolerance(ref), f"step {si_}: logit error {Dall.max()}"
            st = DecodeState.from_host(pre, P, G, G, BLK)
            m.denoise_step(st, Sched(BLK, S), Gate(delta_p, m_req, gate_on, 1))
            gpu = st.to_host()
            p1_all = margins(ref, spec.mask_id) > 2 * Dall                  # P1, every row
            assert (gpu["top1"][0][p1_all] == o["x_hat"][p1_all]).all(), f"step {si_} top-1"
            dlnc = np.abs(np.log(gpu["conf"][0].astype(np.float64)) - np.log(o["c"]))
            assert (dlnc <= 2 * Dall + CONF_RTOL).all(), f"step {si_} confidence"
            ob = dict(o, gamma=margins(ref[lo - P:lo - P + BLK], spec.mask_id),
                      c=o["c"][lo - P:lo - P + BLK])
            dec_ok, p1 = _comparable(ob, pre["unresolved"][0], lo, Dall[lo - P:lo - P + BLK],
                                     delta_p, gate_on)
            # the counter of a block position also needs its whole history certain: teacher
            # forcing gives both sides the same history, so P1 of this step suffices
            want = np.zeros(BLK, np.int64)
            want[np.asarray(o["T"], np.int64) - lo] = 1
            want[np.asarray(o["A"], np.int64) - lo] = 2
            assert (gpu["decision"][0][dec_ok] == want[dec_ok]).all(), f"step {si_} decisions"
            U = pre["unresolved"][0][lo:lo + BLK] == 1
            n_dec += int(U.sum())
            n_dec_ok += int((dec_ok & U).sum())
            nxt = trace[si_ + 1]["pre"] if si_ + 1 < len(trace) else None
            if nxt is None:
                continue
            # counters and previous top-1 of every generation position with a certain top-1
            for n in ("prev_top1", "persist"):
                assert (gpu[n][0][gen][p1_all] == nxt[n][0][gen][p1_all]).all(), \
                    f"step {si_} {n}"
            outside = np.ones(L, bool)
            outside[lo:lo + BLK] = False
            for n in ("tokens", "unresolved"):
                assert (gpu[n][0][outside] == pre[n][0][outside]).all(), f"step {si_} {n}"
    print(f"[summary] global scope, steps {len(trace)}: decisions compared {n_dec_ok}/{n_dec}")
    assert n_dec_ok >= min_frac * n_dec


@pytest.mark.parametrize("delta_p,m_req,gate_on", [(0.65, 1, False), (0.0, 0, True),
                                                   (0.3, 1, True)])
def test_global_scope_block_decode(delta_p, m_req, gate_on):
    """block_decode under the GLOBAL scope equals the GPU's own step-by-step trajectory;
    gate off is the dense decoder, accept-all ends every block in one pass."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = SEPARATED
    prompt = si.prompt_tokens(1, 2, P, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, G, spec.mask_id)
    sched, gate = Sched(BLK, S), Gate(delta_p, m_req, gate_on, 1)
    with Model(spec, seed=0, max_batch=2, max_seq=L) as m:
        st = DecodeState.from_host(host, P, G, G, BLK)
        for _ in range((G // BLK) * S):
            if (st.to_host()["block_idx"] >= G // BLK).all():
                break
            m.denoise_step(st, sched, gate)
        final = st.to_host()
        out, passes, total = m.block_decode(to_dev(prompt), G, sched, gate)
    assert (out.cpu().numpy() == final["tokens"]).all() and (passes == final["passes"]).all()
    assert (final["tokens"][:, P:] != spec.mask_id).all()
    if not gate_on:
        assert (passes == S).all()
    if delta_p <= 0 and m_req == 0:
        assert (passes == 1).all()


@pytest.mark.parametrize("scope", [0, 1])
@pytest.mark.parametrize("delta_p,m_req,gate_on", [(0.65, 1, False), (0.3, 1, True)])
def test_eos_aware_teacher_forced_steps(delta_p, m_req, gate_on, scope):
    """EOS-aware controller (R27), teacher-forced from the oracle's EOS-aware trajectory on
    the separated tiny model; the EOS id is a token of the oracle's fixed-horizon output in
    block 0, so a cut happens.  Decisions are compared where the logit error cannot flip them
    (P1-P3); the removals of a step (decision 3) and the stop are compared where the cut is
    certain: every unresolved block position up to it has a certain decision and top-1."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = SEPARATED
    sc = "global" if scope else "block"
    prompt = si.prompt_tokens(1, 1, P, spec.vocab, spec.mask_id)
    fn = _logits_fn(spec)
    t_fh, _, _ = decode.block_decode(fn, prompt, G, spec.mask_id, BLK, S, delta_p, m_req,
                                     gate_on, scope=sc)
    eos = int(t_fh[0, P + 20])
    _, passes_or, trace = decode.block_decode(fn, prompt, G, spec.mask_id, BLK, S, delta_p,
                                              m_req, gate_on, record=True, scope=sc,
                                              eos_id=eos)
    assert any(s["out"][0]["eos_cut"] is not None for s in trace)
    n_dec = n_ok = cuts_checked = 0
    with Model(spec, seed=0, max_batch=1, max_seq=L) as m:
        for si_, step in enumerate(trace):
            log_case(f"eos-aware teacher-forced step {si_} scope={sc} gate={gate_on}")
            pre, o = step["pre"], step["out"][0]
            lo = P + o["block"] * BLK
            r0 = lo if scope == 0 else P
            n = BLK if scope == 0 else G
            ref = step["logits"][0]
            lg = bf16_to_f32(m.forward_logits(to_dev(pre["tokens"].astype(np.int32)), r0, n)
                             .cpu().numpy())[0].astype(np.float64)
            D = np.max(np.abs(lg - ref), axis=-1)
            assert D.max() <= logit_tolerance(ref)
            st = DecodeState.from_host(pre, P, G, n, BLK)
            m.denoise_step(st, Sched(BLK, S, eos), Gate(delta_p, m_req, gate_on, scope))
            gpu = st.to_host()
            ob = dict(o, gamma=margins(ref[lo - r0:lo - r0 + BLK], spec.mask_id),
                      c=o["c"][lo - r0:lo - r0 + BLK])
            dec_ok, p1 = _comparable(ob, pre["unresolved"][0], lo, D[lo - r0:lo - r0 + BLK],
                                     delta_p, gate_on)
            U = pre["unresolved"][0][lo:lo + BLK] == 1
            want = np.zeros(BLK, np.int64)
            want[np.asarray(o["T"], np.int64) - lo] = 1
            want[np.asarray(o["A"], np.int64) - lo] = 2
            rem = np.asarray(o["removed"], np.int64)
            rem_blk = rem[(rem >= lo) & (rem < lo + BLK)] - lo
            cut = o["eos_cut"]
            end = BLK if cut is None or cut >= lo + BLK else max(cut - lo + 1, 0)
            cut_certain = bool((dec_ok & p1)[:end][U[:end]].all())
            cmp = dec_ok & U
            if not cut_certain:
                cmp[rem_blk] = False
            want[rem_blk] = 3
            assert (gpu["decision"][0][cmp] == want[cmp]).all(), f"step {si_} decisions"
            n_dec += int(U.sum())
            n_ok += int(cmp.sum())
            nxt = trace[si_ + 1]["pre"] if si_ + 1 < len(trace) else None
            if cut is not None and cut_certain and (dec_ok & p1)[U].all() and nxt is not None:
                for k in ("tokens", "unresolved", "block_idx", "step_idx"):
                    assert (gpu[k][0] == nxt[k][0]).all(), f"step {si_} {k}"
                cuts_checked += 1
    print(f"[summary] eos-aware scope={sc}: decisions compared {n_ok}/{n_dec}, "
          f"whole-state checks after a cut {cuts_checked}, oracle passes {passes_or.tolist()}")
    assert n_ok >= 0.3 * n_dec


@pytest.mark.parametrize("scope", [0, 1])
def test_eos_aware_block_decode(scope):
    """block_decode with the EOS-aware controller equals the GPU's own step-by-step
    trajectory; no block after the cut runs and nothing after the cut stays masked."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec = SEPARATED
    prompt = si.prompt_tokens(1, 2, P, spec.vocab, spec.mask_id)
    host = si.initial_decode_state(prompt, G, spec.mask_id)
    gate = Gate(0.3, 1, True, scope)
    with Model(spec, seed=0, max_batch=2, max_seq=L) as m:
        y0, _, _ = m.block_decode(to_dev(prompt), G, Sched(BLK, S), gate)
        eos = int(y0.cpu().numpy()[0, P + 10])
        sched = Sched(BLK, S, eos)
        st = DecodeState.from_host(host, P, G, BLK if scope == 0 else G, BLK)
        for _ in range((G // BLK) * S):
            if (st.to_host()["block_idx"] >= G // BLK).all():
                break
            m.denoise_step(st, sched, gate)
        final = st.to_host()
        out, passes, total = m.block_decode(to_dev(prompt), G, sched, gate)
    y = out.cpu().numpy()
    assert (y == final["tokens"]).all() and (passes == final["passes"]).all()
    gen = y[0, P:]
    cut = int(np.nonzero(gen == eos)[0][0])
    assert (passes[0, cut // BLK + 1:] == 0).all()
    assert (gen != spec.mask_id).all() and (y[1, P:] != spec.mask_id).all()


@pytest.mark.parametrize("scope", [0, 1])
def test_compacted_block_decode(scope):
    """Batch-row compaction: rows cut by the EOS-aware controller finish at different
    passes and leave the dense pass.  On this model no kernel's split of the work depends
    on the row count, so the compacted decode must equal the uncompacted one bit for bit,
    and every row must equal a decode of that row alone."""
    require_gpu()
    from paper_2608_11235_amd import Gate, Model, Sched
    spec = SEPARATED
    B = 3
    prompt = si.prompt_tokens(4, B, P, spec.vocab, spec.mask_id)
    gate = Gate(0.3, 1, True, scope)
    with Model(spec, seed=0, max_batch=B, max_seq=L) as m:
        y0, _, _ = m.block_decode(to_dev(prompt), G, Sched(BLK, S), gate)
        eos = int(y0.cpu().numpy()[0, P + 5])
        sched = Sched(BLK, S, eos)
        out_c, passes_c, total_c = m.block_decode(to_dev(prompt), G, sched, gate)
        m.set_compaction(False)
        out_u, passes_u, total_u = m.block_decode(to_dev(prompt), G, sched, gate)
        m.set_compaction(True)
        alone = [m.block_decode(to_dev(prompt[b:b + 1]), G, sched, gate) for b in range(B)]
    yc, yu = out_c.cpu().numpy(), out_u.cpu().numpy()
    log_case(f"compaction scope={scope}: passes per row {passes_c.sum(1).tolist()}, "
             f"total {total_c}")
    assert (yc == yu).all() and (passes_c == passes_u).all() and total_c == total_u
    rows = passes_c.sum(1)
    assert rows.min() < rows.max(), "rows should finish at different passes"
    for b in range(B):
        assert (alone[b][0].cpu().numpy()[0] == yc[b]).all(), f"row {b} alone"
        assert (alone[b][1][0] == passes_c[b]).all(), f"row {b} passes"
