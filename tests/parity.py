"""Helpers for GPU-vs-oracle parity: tolerances and decision-comparability rules.

Logit tolerance: max |l_gpu - l_oracle| <= 2e-2 * S, with S the logit scale of the compared
rows read shift-invariantly: the softmax of Eq. (1) does not change when a row's logits are
shifted by a constant, so S is the largest per-row range max_v l - min_v l (bf16 GEMMs, fp32
accumulation).

A decision is compared bit-exactly only where the measured per-row logit error D_i cannot
flip it (Proposition 1: an argmax survives any perturbation below half its margin):
  P1 top-1:      oracle margin gamma_i > 2 D_i
  P2 gate:       |ln c_i - ln delta_p| > 2 D_i       (ln c moves by at most 2 D_i)
  P3 transfer:   ln-confidence gap between the k-th and (k+1)-th candidates > 2 (D_a + D_b)
Inputs shared bit-for-bit (vocab/gate kernel alone) have D_i = 0; there the only slack is
the fp32-vs-fp64 rounding of c, covered by CONF_RTOL.
"""
import numpy as np

LOGIT_TOL_FRAC = 2e-2
CONF_RTOL = 2e-5


def bf16_to_f32(bits):
    return (np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16).view(np.float32)


def logit_scale(ref):
    """Largest per-row range (max - min) of the reference logits."""
    ref = np.atleast_2d(np.asarray(ref, dtype=np.float64))
    return float(np.max(ref.max(axis=-1) - ref.min(axis=-1)))


def logit_tolerance(ref):
    return LOGIT_TOL_FRAC * logit_scale(ref)


def margins(logits, mask_id=None):
    l = np.array(logits, dtype=np.float64, copy=True)
    if mask_id is not None:
        l[..., mask_id] = -np.inf
    top2 = np.sort(l, axis=-1)[..., -2:]
    return top2[..., 1] - top2[..., 0]


def comparable_gate(c_or, delta_p, D):
    """P2 on oracle confidences c_or with per-row error bound D (0 for shared inputs)."""
    c = np.asarray(c_or, dtype=np.float64)
    gap = np.abs(np.log(np.maximum(c, 1e-300)) - np.log(delta_p))
    return gap > np.maximum(2 * np.asarray(D), CONF_RTOL)


def comparable_transfer(c_or, cand_rows, k, D):
    """P3: is the top-k split of the candidate rows stable under perturbations D?"""
    if k <= 0 or len(cand_rows) <= k:
        return True
    c = np.asarray(c_or, dtype=np.float64)[cand_rows]
    d = np.asarray(D, dtype=np.float64)
    d = d[cand_rows] if d.ndim else np.full(len(cand_rows), float(d))
    order = np.lexsort((np.asarray(cand_rows), -c))
    a, b = order[k - 1], order[k]
    gap = np.log(c[a]) - np.log(c[b])
    return gap > max(2 * (d[a] + d[b]), CONF_RTOL)
