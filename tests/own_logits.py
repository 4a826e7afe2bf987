"""Decision parity of one GPU denoising step against the oracle's rules run on the GPU's own
logits.

The dense pass is checked against the fp64 oracle elsewhere, within the bf16 logit bound;
there most decisions of a random-init model sit inside that bound and cannot be compared.
Here the oracle's decision rules (Eqs. 1-4, the transfer rule, termination, the EOS-aware
controller) are applied to the very bf16 logits the GPU computes for the pre-step state
(cora_forward_logits on the same rows; the LM-head kernel and every summation order are
planned for the model's max_batch, so a row's logits are the ones the step's batched pass
computes).  Both sides then see identical logits; the only slack left is the fp32 (GPU)
versus fp64 (oracle) rounding of the confidence, so every decision whose cut or threshold is
farther than `rtol` in ln c is compared bit for bit, and so is the state the step writes.
"""
import numpy as np

from oracle import decode
from tests.gpu_common import to_dev
from tests.parity import bf16_to_f32, comparable_decisions

STATE = ("tokens", "unresolved", "prev_top1", "persist", "block_idx", "step_idx")


def conf_rtol(vocab):
    """fp32 sum of exp over the vocabulary (hardware exp2) against fp64: relative error of c."""
    return 2e-5 if vocab <= 4096 else 1e-4


def gpu_rows_logits(m, tokens_row, r0, n):
    """The GPU's bf16 logits of canvas rows [r0, r0 + n) for one batch row, as fp64."""
    out = m.forward_logits(to_dev(np.ascontiguousarray(tokens_row[None, :]).astype(np.int32)),
                           r0, n)
    return bf16_to_f32(out.cpu().numpy())[0].astype(np.float64)


def check_step(m, st_dev, sched, gate, spec, P, G, scope="block", eos_id=None, rtol=None):
    """Run one GPU step on st_dev and compare it with decode.step_row on the GPU's logits.

    Returns (compared, total): unresolved active-block positions whose decision was compared,
    and all of them.  Raises AssertionError on any mismatch."""
    blk, S = sched.block_len, sched.steps_per_block
    n_blocks = G // blk
    rtol = conf_rtol(spec.vocab) if rtol is None else rtol
    pre = st_dev.to_host()
    st_or = {k: pre[k].astype(np.int64) for k in STATE}
    live = [b for b in range(pre["tokens"].shape[0]) if pre["block_idx"][b] < n_blocks]
    outs, logits = {}, {}
    for b in live:
        lo = P + int(pre["block_idx"][b]) * blk
        r0, n = (lo, blk) if scope == "block" else (P, G)
        logits[b] = gpu_rows_logits(m, pre["tokens"][b], r0, n)
        outs[b] = decode.step_row(st_or, b, logits[b], P, blk, S, n_blocks, spec.mask_id,
                                  gate.delta_p, gate.m_req, gate.enabled, logits_row0=r0,
                                  scope=scope, eos_id=eos_id)
    m.denoise_step(st_dev, sched, gate)
    post = st_dev.to_host()
    compared = total = 0
    for b in live:
        o = outs[b]
        lo = P + o["block"] * blk
        off = 0 if scope == "block" else lo - P
        # Eq. (1) on identical logits: top-1 bit-exact (lowest id, mask id left out), c in fp32
        assert (post["top1"][b] == o["x_hat"]).all(), f"row {b}: top-1"
        rel = np.abs(post["conf"][b].astype(np.float64) / o["c"] - 1.0)
        assert (rel <= rtol).all(), f"row {b}: confidence rel err {rel.max():.3g}"
        U = pre["unresolved"][b][lo:lo + blk] == 1
        c_blk = o["c"][off:off + blk]
        # identical logits: the top-1 (asserted equal above) and so the counters are certain
        sure = np.full(blk, np.inf)
        dec_ok, _ = comparable_decisions(c_blk, sure, np.asarray(o["T"]) - lo, o["k"], U, 0.0,
                                         gate.delta_p, gate.enabled, rtol)
        want = np.zeros(blk, np.int64)
        want[np.asarray(o["T"], np.int64) - lo] = 1
        want[np.asarray(o["A"], np.int64) - lo] = 2
        rem = np.asarray(o["removed"], np.int64)
        want[rem[(rem >= lo) & (rem < lo + blk)] - lo] = 3
        certain = bool(dec_ok[U].all())
        cmp = dec_ok & U
        if not certain:
            # an uncertain commit can move the EOS cut: decision 3 is compared only when every
            # decision of the row is certain
            cmp &= (want != 3) & (post["decision"][b] != 3)
        got = post["decision"][b].astype(np.int64)
        assert (got[cmp] == want[cmp]).all(), \
            f"row {b}: decisions {got[cmp]} != {want[cmp]} at {np.nonzero(cmp)[0]}"
        compared += int(cmp.sum())
        total += int(U.sum())
        if certain:
            # every decision certain: the whole post-step state of the row is the oracle's
            for k in STATE:
                assert (np.asarray(post[k][b]) == np.asarray(st_or[k][b])).all(), \
                    f"row {b}: state {k}"
            assert int(post["done"][b]) == int(o["done"]), f"row {b}: done"
        else:
            # positions outside the active block keep their values, apart from the GLOBAL
            # scope's counters and an EOS cut's removals, which need certain decisions
            outside = np.ones(pre["tokens"].shape[1], bool)
            outside[lo:lo + blk] = False
            if eos_id is None:
                names = ("tokens", "unresolved") if scope == "global" else STATE[:4]
                for k in names:
                    assert (post[k][b][outside] == st_or[k][b][outside]).all(), f"row {b}: {k}"
    return compared, total


def run_decode(m, st_dev, sched, gate, spec, P, G, scope="block", eos_id=None, max_steps=None):
    """Step the GPU's own trajectory to the end (or max_steps), checking every step."""
    n_blocks = G // sched.block_len
    compared = total = steps = 0
    while (st_dev.block_idx.cpu().numpy() < n_blocks).any():
        if max_steps is not None and steps >= max_steps:
            break
        c, t = check_step(m, st_dev, sched, gate, spec, P, G, scope, eos_id)
        compared += c
        total += t
        steps += 1
    return compared, total, steps
