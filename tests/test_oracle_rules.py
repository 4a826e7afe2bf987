"""Pins of the oracle's decision rules and gated block decode (Eqs. 2-4, termination).

Against: a hand-worked decode (tests/golden/worked_example.json), invariants the
paper states (U shrinks by exactly T and A, committed tokens never change, the
gate acts only on positions the transfer rule leaves, dense recovery with the
gate off), and special cases with known pass counts.
"""
import json
import os

import numpy as np
import pytest

from oracle import decode, theory


def test_persistence_counter_scripted():
    """Eq. (2): counter zero at the first executed step, +1 per repeated top-1, reset on change."""
    seq = [5, 5, 7, 7, 7, 2, 2]
    want = [0, 1, 0, 1, 2, 0, 1]
    prev, m = np.array([decode.NONE]), np.array([0])
    got = []
    for x in seq:
        prev, m = decode.persistence_update(prev, m, np.array([x]))
        got.append(int(m[0]))
    assert got == want


def test_transfer_schedule():
    assert decode.transfer_schedule(32, 16).tolist() == [2] * 16
    assert decode.transfer_schedule(32, 32).tolist() == [1] * 32
    assert decode.transfer_schedule(10, 4).tolist() == [3, 3, 2, 2]
    for M in range(1, 40):
        for S in range(1, M + 1):
            k = decode.transfer_schedule(M, S)
            assert k.sum() == M and k.max() - k.min() <= 1 and (np.diff(k) <= 0).all()


def test_transfer_set_ties_and_clipping():
    c32 = np.zeros(10, np.float32)
    c32[[2, 5, 7]] = [0.5, 0.9, 0.5]
    assert decode.transfer_set([2, 5, 7], c32, 1).tolist() == [5]
    assert decode.transfer_set([2, 5, 7], c32, 2).tolist() == [2, 5]     # tie 2 vs 7 -> 2
    assert decode.transfer_set([2, 5, 7], c32, 9).tolist() == [2, 5, 7]
    assert decode.transfer_set([], c32, 3).tolist() == []


def test_gate_inclusive_boundaries():
    c = np.array([0.5, 0.5, np.nextafter(np.float32(0.5), np.float32(0))], np.float32)
    m = np.array([1, 0, 1])
    assert decode.gate_accept(c, m, 0.5, 1).tolist() == [True, False, False]
    assert decode.gate_accept(c, m, 0.5, 0).tolist() == [True, True, False]


def _scripted_logits_fn(script, V):
    calls = {"n": 0}

    def fn(tokens, rows):
        s = calls["n"]
        calls["n"] += 1
        out = []
        for b, r in enumerate(rows):
            l = np.zeros((len(r), V))
            for j, p in enumerate(r):
                if str(int(p)) in script[s]:
                    l[j] = script[s][str(int(p))]
            out.append(l)
        return out
    return fn


def test_worked_example(golden_dir):
    with open(os.path.join(golden_dir, "worked_example.json")) as f:
        ex = json.load(f)
    for case in ex["cases"]:
        fn = _scripted_logits_fn(ex["script"], ex["vocab"])
        tokens, passes, trace = decode.block_decode(
            fn, np.array(ex["prompt"]), ex["gen_len"], ex["mask_id"], ex["block_len"],
            ex["steps_per_block"], case["delta_p"], case["m_req"], case["gate_enabled"],
            record=True)
        assert tokens.tolist() == case["tokens"], case["name"]
        assert passes.tolist() == case["passes"], case["name"]
        for want, step in zip(case["per_step"], trace):
            out = step["out"][0]
            assert out["T"].tolist() == want["T"], case["name"]
            assert out["A"].tolist() == want["A"], case["name"]


class _RandomModel:
    """Deterministic stand-in backbone: logits are a fixed random function of the canvas,
    so earlier commits change later predictions (accepted tokens stay visible)."""

    def __init__(self, V, L, seed, scale):
        rng = np.random.default_rng(seed)
        self.E = rng.normal(0, 1, (V, 16))
        self.P = rng.normal(0, 1, (L, 16))
        self.W = rng.normal(0, 1, (16, V)) * scale
        self.V = V

    def __call__(self, tokens, rows):
        out = []
        for b, r in enumerate(rows):
            ctx = np.tanh(self.E[tokens[b]].mean(0))
            h = self.P[np.asarray(r)] + ctx
            out.append(h @ self.W)
        return out


@pytest.mark.parametrize("scope", ["block", "global"])
@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("delta_p,m_req,gate", [(0.65, 1, True), (0.3, 0, True), (0.5, 2, True),
                                                 (0.0, 1, True), (0.65, 1, False)])
def test_decode_invariants(seed, delta_p, m_req, gate, scope):
    """(0.0, 1) is the persistence-only variant, (0.3, 0) confidence-only, m = 2 two checks."""
    _check_decode_invariants(seed, delta_p, m_req, gate, scope, 23, 5, 24, 8, 4)


@pytest.mark.parametrize("scope", ["block", "global"])
@pytest.mark.parametrize("seed", range(2))
@pytest.mark.parametrize("delta_p,m_req,gate", [(0.65, 1, True), (0.3, 0, True), (0.5, 2, True),
                                                 (0.0, 1, True), (0.65, 1, False)])
@pytest.mark.parametrize("P,G,blk,S", [(0, 24, 8, 4),     # empty prompt
                                       (5, 6, 1, 1),      # one-position blocks
                                       (3, 32, 32, 32),   # one block, one transfer per step
                                       (2, 16, 16, 3)])   # k_s = 6, 5, 5
def test_decode_invariants_degenerate_shapes(seed, delta_p, m_req, gate, scope, P, G, blk, S):
    _check_decode_invariants(seed, delta_p, m_req, gate, scope, 23, P, G, blk, S)


def _check_decode_invariants(seed, delta_p, m_req, gate, scope, V, P, G, blk, S):
    mask_id = V - 1
    model = _RandomModel(V, P + G, seed, scale=1.5)
    prompt = np.random.default_rng(100 + seed).integers(0, V - 1, (2, P))
    tokens, passes, trace = decode.block_decode(model, prompt, G, mask_id, blk, S, delta_p,
                                                m_req, gate, record=True, scope=scope)
    ks = decode.transfer_schedule(blk, S)
    for step in trace:
        pre = step["pre"]
        for b, out in step["out"].items():
            lo = P + out["block"] * blk
            pos = np.arange(lo, lo + blk)
            U_blk = pos[pre["unresolved"][b, pos] == 1]
            T, A = out["T"], out["A"]
            assert len(np.intersect1d(T, A)) == 0                  # gate only on U \ T
            assert set(T) <= set(U_blk) and set(A) <= set(U_blk)   # only the active block
            assert len(T) == min(ks[out["step"]], len(U_blk))      # exactly k_s fixed
            row0 = lo if scope == "block" else P
            for i in A:                                            # Eq. (3)
                assert out["c32"][i - row0] >= np.float32(delta_p) and out["m"][i] >= m_req
            if not gate:
                assert len(A) == 0
            # T holds the highest confidences of U_blk
            if len(T) and len(U_blk) > len(T):
                rest = np.setdiff1d(U_blk, T)
                assert out["c32"][T - row0].min() >= out["c32"][rest - row0].max()
    # Eq. (4): U shrinks by exactly T and A, committed tokens never change afterwards
    for s0, s1 in zip(trace[:-1], trace[1:]):
        for b, out in s0["out"].items():
            fixed = np.union1d(out["T"], out["A"])
            before, after = s0["pre"]["unresolved"][b], s1["pre"]["unresolved"][b]
            assert (before.astype(int) - after.astype(int)).sum() == len(fixed)
            assert (after[fixed] == 0).all()
            committed = np.where(before == 0)[0]
            assert (s1["pre"]["tokens"][b, committed] == s0["pre"]["tokens"][b, committed]).all()
    assert (tokens != mask_id).all()
    if not gate:
        assert (passes == S).all()                                   # dense horizon
    elif m_req >= 1 and scope == "block":
        assert (passes >= min(m_req + 1, S)).all()                   # persistence needs repeats
    elif m_req >= 1:
        assert (passes[:, 0] >= min(m_req + 1, S)).all()             # first block: no history
    assert 0.0 <= theory.step_ratio(passes, np.full_like(passes, S)) <= 1.0


@pytest.mark.parametrize("seed", range(4))
def test_gate_off_equals_unreachable_threshold(seed):
    """Dense recovery: with the gate disabled the decoder is the original one, which is the
    same as a threshold no confidence can reach (c <= 1 < 1.5)."""
    V, P, G, blk, S = 19, 4, 16, 8, 8
    model = _RandomModel(V, P + G, seed, scale=3.0)
    prompt = np.random.default_rng(seed).integers(0, V - 1, (1, P))
    t_off, p_off, _ = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.65, 1, False)
    t_hi, p_hi, _ = decode.block_decode(model, prompt, G, V - 1, blk, S, 1.5, 0, True)
    t_end, p_end = decode.dense_endpoint(model, prompt, G, V - 1, blk, S)
    assert (t_off == t_hi).all() and (p_off == p_hi).all() and (t_off == t_end).all()
    assert (p_end == S).all()


def test_accept_all_ends_each_block_in_one_pass():
    V, P, G, blk, S = 17, 3, 32, 8, 8
    model = _RandomModel(V, P + G, 7, scale=1.0)
    prompt = np.zeros((2, P), dtype=np.int64)
    _, passes, _ = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.0, 0, True)
    assert (passes == 1).all()


def test_batch_rows_are_independent():
    V, P, G, blk, S = 29, 4, 16, 8, 4
    model = _RandomModel(V, P + G, 3, scale=4.0)
    prompt = np.random.default_rng(9).integers(0, V - 1, (3, P))
    t_all, p_all, _ = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.4, 1, True)
    for b in range(3):
        t1, p1, _ = decode.block_decode(model, prompt[b:b + 1], G, V - 1, blk, S, 0.4, 1, True)
        assert (t1[0] == t_all[b]).all() and (p1[0] == p_all[b]).all()


@pytest.mark.parametrize("seed", range(4))
def test_global_scope_gate_off_is_dense(seed):
    """R5 only changes what the gate sees: with the gate off both scopes are the original
    decoder (dense endpoint, S passes per block)."""
    V, P, G, blk, S = 19, 4, 16, 8, 8
    model = _RandomModel(V, P + G, seed, scale=3.0)
    prompt = np.random.default_rng(seed).integers(0, V - 1, (1, P))
    t_g, p_g, _ = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.65, 1, False,
                                      scope="global")
    t_end, p_end = decode.dense_endpoint(model, prompt, G, V - 1, blk, S)
    assert (t_g == t_end).all() and (p_g == p_end).all()


@pytest.mark.parametrize("seed", range(4))
def test_global_counters_dominate_block(seed):
    """On one trajectory (gate off, so both scopes decode identically) the GLOBAL counter of
    an active-block position is never below its BLOCK counter: BLOCK restarts it at the
    block's first executed step, GLOBAL has counted since the position's first pass."""
    V, P, G, blk, S = 13, 3, 24, 8, 4
    model = _RandomModel(V, P + G, seed, scale=0.7)
    prompt = np.random.default_rng(seed).integers(0, V - 1, (1, P))
    _, _, tr_b = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.65, 1, False,
                                     record=True, scope="block")
    _, _, tr_g = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.65, 1, False,
                                     record=True, scope="global")
    assert len(tr_b) == len(tr_g)
    strictly = 0
    for sb, sg in zip(tr_b, tr_g):
        ob, og = sb["out"][0], sg["out"][0]
        lo = P + ob["block"] * blk
        pos = np.arange(lo, lo + blk)
        U = pos[sb["pre"]["unresolved"][0, pos] == 1]
        assert (og["m"][U] >= ob["m"][U]).all()
        strictly += int((og["m"][U] > ob["m"][U]).sum())
    assert strictly > 0   # later blocks did inherit history


def test_global_scope_worked_example():
    """Hand-worked (R5): V = 3 (tokens 0, 1; mask 2), prompt 1, gen 4, blocks of 2, S = 2
    (k_s = 1, 1), delta_p 0.6, m = 1.  Every position's logits are (4, 0, -) on every pass:
    top-1 token 0 with c = e^4 / (e^4 + 1) = 0.982, equal confidences -> lower position.
      BLOCK: each block starts with fresh counters: pass 1 fixes its first position by the
      transfer rule (the other has m = 0), pass 2 transfers the second -> passes (2, 2).
      GLOBAL: positions 3, 4 are scored from pass 1: after passes 1-2 their counters are 1;
      pass 3 (block 1, m = 2) transfers 3 and the gate accepts 4 -> passes (2, 1)."""
    V, mask = 3, 2

    def fn(tokens, rows):
        return [np.tile(np.array([4.0, 0.0, 0.0]), (len(r), 1)) for r in rows]

    prompt = np.array([[1]])
    t_b, p_b, tr_b = decode.block_decode(fn, prompt, 4, mask, 2, 2, 0.6, 1, True, record=True,
                                         scope="block")
    t_g, p_g, tr_g = decode.block_decode(fn, prompt, 4, mask, 2, 2, 0.6, 1, True, record=True,
                                         scope="global")
    assert p_b.tolist() == [[2, 2]] and p_g.tolist() == [[2, 1]]
    assert t_b.tolist() == [[1, 0, 0, 0, 0]] and t_g.tolist() == [[1, 0, 0, 0, 0]]
    assert [o["out"][0]["T"].tolist() for o in tr_g] == [[1], [2], [3]]
    assert [o["out"][0]["A"].tolist() for o in tr_g] == [[], [], [4]]
    assert tr_g[2]["out"][0]["m"][4] == 2 and tr_b[3]["out"][0]["m"][4] == 1


def _eotp_script_fn(logit_of_pos, V):
    """Every pass: position p's logits are fixed (token, logit) pairs, other entries 0."""
    def fn(tokens, rows):
        out = []
        for r in rows:
            l = np.zeros((len(r), V))
            for j, p in enumerate(r):
                for tok, val in logit_of_pos.get(int(p), []):
                    l[j, tok] = val
            out.append(l)
        return out
    return fn


def test_eotp_worked_example():
    """Hand-worked (R27): V = 4 (tokens 0, 1; EOS 2; mask 3), prompt 1, gen 6, blocks of 2,
    S = 2 (k_s = 1, 1).  Position 1 -> token 0 (logit 3, c = e^3/(e^3+2) = 0.909),
    position 2 -> EOS (logit 5, c = 0.987), position 3 -> token 1 (logit 4), 4-6 -> token 0
    (logit 2).
      fixed horizon, gate off: every block takes 2 passes; output 0 EOS 1 0 0 0.
      EoTP, gate off: pass 1 transfers the EOS at 2 (highest c) -> positions 3-6 become EOS;
        pass 2 transfers position 1 -> block done, row stops: passes (2, 0, 0).
      EoTP, gate (0.6, m = 0): pass 1 transfers the EOS and accepts position 1 -> (1, 0, 0)."""
    V, EOS, MASK = 4, 2, 3
    script = {1: [(0, 3.0)], 2: [(EOS, 5.0)], 3: [(1, 4.0)], 4: [(0, 2.0)], 5: [(0, 2.0)],
              6: [(0, 2.0)]}
    fn = _eotp_script_fn(script, V)
    prompt = np.array([[1]])
    t, p, _ = decode.block_decode(fn, prompt, 6, MASK, 2, 2, 0.6, 0, False)
    assert p.tolist() == [[2, 2, 2]] and t.tolist() == [[1, 0, EOS, 1, 0, 0, 0]]
    t, p, tr = decode.block_decode(fn, prompt, 6, MASK, 2, 2, 0.6, 0, False, record=True,
                                   eos_id=EOS)
    assert p.tolist() == [[2, 0, 0]] and t.tolist() == [[1, 0, EOS, EOS, EOS, EOS, EOS]]
    assert tr[0]["out"][0]["eos_cut"] == 2 and tr[0]["out"][0]["removed"].tolist() == [3, 4, 5, 6]
    t, p, _ = decode.block_decode(fn, prompt, 6, MASK, 2, 2, 0.6, 0, True, eos_id=EOS)
    assert p.tolist() == [[1, 0, 0]] and t.tolist() == [[1, 0, EOS, EOS, EOS, EOS, EOS]]


@pytest.mark.parametrize("gate", [False, True])
@pytest.mark.parametrize("seed", range(5))
def test_eotp_follows_fixed_horizon_until_eos(seed, gate):
    """Until the step that commits the first EOS, the EOS-aware decode is the fixed-horizon
    one; afterwards no later block runs and every later position is EOS unless it was
    committed before the cut.  The EOS id is taken from the fixed-horizon output so it
    occurs."""
    V, P, G, blk, S = 17, 3, 32, 8, 4
    model = _RandomModel(V, P + G, seed, scale=2.0)
    prompt = np.random.default_rng(seed).integers(0, V - 1, (1, P))
    t_fh, p_fh, tr_fh = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.5, 1, gate,
                                            record=True)
    eos = int(t_fh[0, P + G // 2])
    t_e, p_e, tr_e = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.5, 1, gate,
                                         record=True, eos_id=eos)
    first = next(i for i, s in enumerate(tr_e) if s["out"][0]["eos_cut"] is not None)
    for a, b in zip(tr_fh[:first + 1], tr_e[:first + 1]):   # same states and decisions
        assert (a["pre"]["tokens"] == b["pre"]["tokens"]).all()
        assert a["out"][0]["T"].tolist() == b["out"][0]["T"].tolist()
        assert a["out"][0]["A"].tolist() == b["out"][0]["A"].tolist()
    cut = tr_e[-1]["out"][0]["eos_cut"]
    assert t_e[0, cut] == eos and not (t_e[0, P:cut] == eos).any()
    cut_blk = (cut - P) // blk
    assert (p_e[0, cut_blk + 1:] == 0).all() and (p_e[0, :cut_blk] == p_fh[0, :cut_blk]).all()
    pre_cut = tr_e[first]["pre"]
    committed = pre_cut["unresolved"][0] == 0
    for i in range(cut + 1, P + G):
        assert t_e[0, i] == eos or committed[i] or i in np.union1d(
            tr_e[first]["out"][0]["T"], tr_e[first]["out"][0]["A"])
    assert p_e.sum() <= p_fh.sum()


def test_eotp_unpredictable_eos_is_fixed_horizon():
    """An EOS id that is never predicted (the mask id) leaves the decoder unchanged."""
    V, P, G, blk, S = 13, 2, 16, 8, 4
    model = _RandomModel(V, P + G, 1, scale=2.0)
    prompt = np.random.default_rng(1).integers(0, V - 1, (2, P))
    a = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.4, 1, True)
    b = decode.block_decode(model, prompt, G, V - 1, blk, S, 0.4, 1, True, eos_id=V - 1)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all()
