"""Oracle of the paper's analysis quantities (test infrastructure only).

Proposition 1 (endpoint-preservation condition), g(delta_p) of Section 3
("Population Disagreement and Calibration"), the prompt step ratio rho, and the
accepted-token and final-output disagreement losses (Eqs. 7 and 12).
"""
import numpy as np


def margin(logits, v=None):
    """gamma = l_v - max_{u != v} l_u for v = the top-1 token (or the given v)."""
    l = np.asarray(logits, dtype=np.float64)
    if v is None:
        v = int(np.argmax(l))
    others = np.delete(l, v)
    return float(l[v] - np.max(others))


def margin_condition_holds(ref_logits, cur_logits):
    """Eq. (5): ||l* - l^(s)||_inf < gamma^(s) / 2 (gamma of the current logits)."""
    d = np.max(np.abs(np.asarray(ref_logits, np.float64) - np.asarray(cur_logits, np.float64)))
    return bool(d < margin(cur_logits) / 2.0)


def confidence_margin_lower_bound(c):
    """Proposition 1, second part: for c > 1/2, gamma >= log(c / (1 - c))."""
    c = np.asarray(c, dtype=np.float64)
    return np.log(c / (1.0 - c))


def g(delta_p):
    """g(delta_p) = 1/2 log(delta_p / (1 - delta_p)) (drift radius in Section 3)."""
    return 0.5 * np.log(delta_p / (1.0 - delta_p))


def step_ratio(passes_h, passes_dense):
    """rho_Q(h) = sum_b S^h_b / sum_b S^dense_b (Section 3, calibration selector)."""
    return float(np.sum(passes_h)) / float(np.sum(passes_dense))


def accepted_disagreement(accepted_positions, accepted_tokens, endpoint):
    """L^acc (Eq. 7): fraction of accepted positions whose accepted token differs from the
    dense endpoint; zero when nothing was accepted."""
    n = len(accepted_positions)
    if n == 0:
        return 0.0
    endpoint = np.asarray(endpoint)
    bad = sum(int(t != endpoint[i]) for i, t in zip(accepted_positions, accepted_tokens))
    return bad / max(1, n)


def output_disagreement(output_gen, endpoint_gen):
    """L^out (Eq. 12): fraction of the n_Q generation positions whose final token differs."""
    a, b = np.asarray(output_gen), np.asarray(endpoint_gen)
    return float(np.mean(a != b))
