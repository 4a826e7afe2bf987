"""The oracle's pins catch plausible mistakes (CPU only).

Each case plants one mistake in the oracle (monkeypatched for that case only): a dropped
term, a wrong sign or index, a transposed operand, a wrong tie-break or comparison.  The
existing pins (tests/test_oracle_forward.py, test_oracle_scores.py, test_oracle_rules.py)
are then run against the planted oracle, and at least one of them must fail.  A mistake no
pin notices would mean the oracle is pinned only where it is already right.
"""
import numpy as np
import pytest

from oracle import decode, theory
from oracle import forward as of
from tests import test_oracle_forward as tf
from tests import test_oracle_rules as tr
from tests import test_oracle_scores as ts


def _pins(golden_dir):
    """Every pin as a zero-argument callable (parametrised pins at representative values)."""
    p = []
    for kw in ({}, {"n_kv_heads": 2, "qkv_bias": True}, {"n_kv_heads": 1}):
        p.append(lambda kw=kw: tf.test_forward_matches_torch_library(kw))
    p += [tf.test_rope_relative_position_identity, tf.test_attention_closed_forms,
          tf.test_rmsnorm_silu_closed_forms]
    for mid in (None, 0, 3):
        p.append(lambda mid=mid: ts.test_top1_confidence_brute_force(mid))
    p += [ts.test_top1_ties_lowest_id, ts.test_confidence_closed_forms,
          ts.test_mask_column_never_predicted, ts.test_prop1_confidence_bounds_margin,
          ts.test_prop1_margin_condition_preserves_argmax_and_is_tight,
          lambda: ts.test_g_of_delta_p_matches_paper(golden_dir),
          ts.test_disagreement_losses_and_ratio]
    p += [tr.test_persistence_counter_scripted, tr.test_transfer_schedule,
          tr.test_transfer_set_ties_and_clipping, tr.test_gate_inclusive_boundaries,
          lambda: tr.test_worked_example(golden_dir)]
    for args in ((0, 0.65, 1, True, "block"), (1, 0.3, 0, True, "global"),
                 (2, 0.5, 2, True, "block"), (3, 0.65, 1, False, "block")):
        p.append(lambda a=args: tr.test_decode_invariants(*a))
    p += [lambda: tr.test_gate_off_equals_unreachable_threshold(0),
          tr.test_accept_all_ends_each_block_in_one_pass, tr.test_batch_rows_are_independent,
          tr.test_global_scope_worked_example, tr.test_eotp_worked_example]
    return p


# ---- planted mistakes ---------------------------------------------------------------------
def _rope_sign(x, cos, sin):
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos + x2 * sin, x2 * cos - x1 * sin], axis=-1)


def _rope_interleaved(x, cos, sin):
    x1, x2 = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2], out[..., 1::2] = x1 * cos - x2 * sin, x2 * cos + x1 * sin
    return out


def _rope_tables_freq(L, hd, theta, dtype=np.float64):
    j = np.arange(hd // 2, dtype=np.float64)
    ang = np.arange(L, dtype=np.float64)[:, None] * (theta ** (-j / hd))[None, :]
    return np.cos(ang).astype(dtype), np.sin(ang).astype(dtype)


def _attention_variant(scale_fn=None, causal=False, kv_of=None):
    def attention(q, k, v):
        H, L, hd = q.shape
        Hkv = k.shape[0]
        out = np.empty_like(q)
        for j in range(H):
            kv = kv_of(j, H, Hkv) if kv_of else j // (H // Hkv)
            s = (q[j] @ k[kv].T) * (scale_fn(hd) if scale_fn else 1.0 / np.sqrt(hd))
            if causal:
                s = np.where(np.tril(np.ones((L, L), bool)), s, -np.inf)
            out[j] = of.softmax(s) @ v[kv]
        return out
    return attention


def _layer_variant(swap_gate_up=False, drop_attn_residual=False, untransposed_q=False):
    def layer_forward(h, w, spec, cos, sin, dtype):
        L, d = h.shape
        H, Hkv, hd = spec.n_heads, spec.n_kv_heads, spec.head_dim
        W = lambda n: np.asarray(w[n], dtype=dtype)  # noqa: E731
        a = of.rmsnorm(h, W("attn_norm"), spec.rms_eps)
        q = a @ (W("wq") if untransposed_q else W("wq").T)
        k, v = a @ W("wk").T, a @ W("wv").T
        if spec.qkv_bias:
            q, k, v = q + W("bq"), k + W("bk"), v + W("bv")
        q = q.reshape(L, H, hd).transpose(1, 0, 2)
        k = k.reshape(L, Hkv, hd).transpose(1, 0, 2)
        v = v.reshape(L, Hkv, hd).transpose(1, 0, 2)
        q, k = of.rope(q, cos, sin), of.rope(k, cos, sin)
        o = of.attention(q, k, v).transpose(1, 0, 2).reshape(L, H * hd)
        h = (o @ W("wo").T) if drop_attn_residual else h + o @ W("wo").T
        a = of.rmsnorm(h, W("mlp_norm"), spec.rms_eps)
        g, u = a @ W("wg").T, a @ W("wu").T
        if swap_gate_up:
            g, u = u, g
        return h + (of.silu(g) * u) @ W("wd").T
    return layer_forward


def _logits_no_scale(weights, spec, h_rows, dtype=np.float64):
    y = of.rmsnorm(h_rows, np.asarray(weights.final_norm, dtype=dtype), spec.rms_eps)
    return y @ np.asarray(weights.lm_head(), dtype=dtype).T


def _top1_variant(highest_tie=False, keep_mask=False, temperature=1.0):
    def top1_confidence(logits, mask_id=None):
        l = np.array(logits, dtype=np.float64, copy=True)
        if mask_id is not None and not keep_mask:
            l[..., mask_id] = -np.inf
        p = np.exp((l - np.max(l, axis=-1, keepdims=True)) / temperature)
        p = p / np.sum(p, axis=-1, keepdims=True)
        if highest_tie:
            V = p.shape[-1]
            x_hat = V - 1 - np.argmax(p[..., ::-1], axis=-1)
        else:
            x_hat = np.argmax(p, axis=-1)
        c = np.take_along_axis(p, x_hat[..., None], axis=-1)[..., 0]
        return x_hat.astype(np.int64), c
    return top1_confidence


def _persist_no_reset(prev, m, x_hat):
    return np.asarray(x_hat).copy(), np.where(prev != decode.NONE, m + 1, 0)


def _persist_counts_first(prev, m, x_hat):
    same = (prev == decode.NONE) | (prev == x_hat)
    return np.asarray(x_hat).copy(), np.where(same, m + 1, 0)


def _schedule_remainder_last(M, S):
    base, rem = divmod(int(M), int(S))
    return np.array([base + (1 if s >= S - rem else 0) for s in range(S)], dtype=np.int64)


def _transfer_variant(lowest=False, later_tie=False):
    def transfer_set(candidates, c32, k):
        candidates = np.asarray(candidates)
        if len(candidates) == 0 or k <= 0:
            return np.zeros(0, dtype=np.int64)
        sgn = 1.0 if lowest else -1.0
        order = sorted(candidates.tolist(),
                       key=lambda i: (sgn * float(c32[i]), -i if later_tie else i))
        return np.array(sorted(order[:min(int(k), len(order))]), dtype=np.int64)
    return transfer_set


def _gate_strict_c(c32, m, delta_p, m_req):
    return (np.asarray(c32, np.float32) > np.float32(delta_p)) & (np.asarray(m) >= m_req)


def _gate_strict_m(c32, m, delta_p, m_req):
    return (np.asarray(c32, np.float32) >= np.float32(delta_p)) & (np.asarray(m) > m_req)


def _gate_or(c32, m, delta_p, m_req):
    return (np.asarray(c32, np.float32) >= np.float32(delta_p)) | (np.asarray(m) >= m_req)


def _gate_ignores_m(c32, m, delta_p, m_req):
    return np.asarray(c32, np.float32) >= np.float32(delta_p)


MUTANTS = {
    "rope sign of the sine term": (of, "rope", _rope_sign),
    "rope pairs (2j, 2j+1) instead of (j, j+hd/2)": (of, "rope", _rope_interleaved),
    "rope frequency theta^(-j/hd)": (of, "rope_tables", _rope_tables_freq),
    "attention without 1/sqrt(hd)": (of, "attention", _attention_variant(scale_fn=lambda hd: 1.0)),
    "attention scaled by 1/hd": (of, "attention", _attention_variant(scale_fn=lambda hd: 1.0 / hd)),
    "causal mask in bidirectional attention": (of, "attention", _attention_variant(causal=True)),
    "GQA kv head j % Hkv": (of, "attention",
                            _attention_variant(kv_of=lambda j, H, Hkv: j % Hkv)),
    "rmsnorm eps outside the root": (of, "rmsnorm",
                                     lambda x, w, eps: x / (np.sqrt(np.mean(x * x, -1, keepdims=True)) + eps) * w),
    "rmsnorm over sum instead of mean": (of, "rmsnorm",
                                         lambda x, w, eps: x / np.sqrt(np.sum(x * x, -1, keepdims=True) + eps) * w),
    "rmsnorm weight dropped": (of, "rmsnorm",
                               lambda x, w, eps: x / np.sqrt(np.mean(x * x, -1, keepdims=True) + eps)),
    "silu replaced by sigmoid": (of, "silu", lambda x: 1.0 / (1.0 + np.exp(-x))),
    "SwiGLU gate and up swapped": (of, "layer_forward", _layer_variant(swap_gate_up=True)),
    "attention residual dropped": (of, "layer_forward", _layer_variant(drop_attn_residual=True)),
    "q projection not transposed": (of, "layer_forward", _layer_variant(untransposed_q=True)),
    "logit scale dropped": (of, "logits_from_hidden", _logits_no_scale),
    "top-1 ties to the highest id": (decode, "top1_confidence", _top1_variant(highest_tie=True)),
    "mask column not excluded": (decode, "top1_confidence", _top1_variant(keep_mask=True)),
    "softmax at temperature 2": (decode, "top1_confidence", _top1_variant(temperature=2.0)),
    "persistence counter never resets": (decode, "persistence_update", _persist_no_reset),
    "persistence counter counts the first step": (decode, "persistence_update",
                                                  _persist_counts_first),
    "schedule remainder on the last steps": (decode, "transfer_schedule",
                                             _schedule_remainder_last),
    "transfer rule takes the lowest confidences": (decode, "transfer_set",
                                                   _transfer_variant(lowest=True)),
    "transfer ties to the higher position": (decode, "transfer_set",
                                             _transfer_variant(later_tie=True)),
    "gate confidence test strict": (decode, "gate_accept", _gate_strict_c),
    "gate persistence test strict": (decode, "gate_accept", _gate_strict_m),
    "gate conjunction read as or": (decode, "gate_accept", _gate_or),
    "gate ignores persistence": (decode, "gate_accept", _gate_ignores_m),
    "g(delta_p) without the factor 1/2": (theory, "g", lambda dp: np.log(dp / (1.0 - dp))),
    "L_acc counts agreements": (theory, "accepted_disagreement",
                                lambda pos, tok, Y: (sum(int(t == np.asarray(Y)[i]) for i, t in
                                                         zip(pos, tok)) / len(pos)) if len(pos) else 0.0),
}


def test_pins_pass_on_the_unplanted_oracle(golden_dir):
    for pin in _pins(golden_dir):
        pin()


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistake_is_caught(name, golden_dir, monkeypatch):
    module, attr, fn = MUTANTS[name]
    caught = []
    with monkeypatch.context() as mp:
        mp.setattr(module, attr, fn)
        for i, pin in enumerate(_pins(golden_dir)):
            try:
                with np.errstate(all="ignore"):
                    pin()
            except Exception:  # an assertion, or the planted oracle breaking a shape
                caught.append(i)
    assert caught, f"no pin notices the planted mistake: {name}"
