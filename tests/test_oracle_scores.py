"""Pins of the oracle's scoring (Eq. 1) and of Proposition 1 / g(delta_p).

Each check compares the oracle with something other than itself: brute-force
enumeration, scipy's softmax, closed forms, or values printed in the paper.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy.special import softmax as sp_softmax

from oracle import decode, theory


def _brute_top1(row, mask_id):
    """Scan in index order keeping the first strict maximum; mask column skipped."""
    best, arg = -math.inf, None
    for i, v in enumerate(row):
        if i == mask_id:
            continue
        if v > best:
            best, arg = v, i
    return arg


@pytest.mark.parametrize("mask_id", [None, 0, 3])
def test_top1_confidence_brute_force(mask_id):
    grid = [-1.0, 0.0, 0.5, 2.0]
    V = 4
    rows = np.array(list(itertools.product(grid, repeat=V)))
    x_hat, c = decode.top1_confidence(rows, mask_id)
    for r, xh, cc in zip(rows, x_hat, c):
        keep = [i for i in range(V) if i != mask_id]
        p = sp_softmax(r[keep])
        assert xh == _brute_top1(r, mask_id if mask_id is not None else -1)
        assert cc == pytest.approx(p.max(), rel=1e-12)


def test_top1_ties_lowest_id():
    row = np.array([[1.0, 3.0, 3.0, 3.0, 0.0]])
    x_hat, c = decode.top1_confidence(row)
    assert x_hat[0] == 1
    # three tied maxima -> c = e^3 / (3 e^3 + e + 1)
    assert c[0] == pytest.approx(math.exp(3) / (3 * math.exp(3) + math.e + 1), rel=1e-13)


def test_confidence_closed_forms():
    for V in (2, 7, 2048):
        x_hat, c = decode.top1_confidence(np.zeros((1, V)))
        assert x_hat[0] == 0 and c[0] == pytest.approx(1.0 / V, rel=1e-13)
        for delta in (0.1, 1.0, 5.0):
            row = np.zeros((1, V))
            row[0, V // 2] = delta
            x_hat, c = decode.top1_confidence(row)
            assert x_hat[0] == V // 2
            assert c[0] == pytest.approx(1.0 / (1.0 + (V - 1) * math.exp(-delta)), rel=1e-12)


def test_mask_column_never_predicted():
    row = np.array([[0.0, 1.0, 50.0, 2.0]])
    x_hat, c = decode.top1_confidence(row, mask_id=2)
    assert x_hat[0] == 3
    assert c[0] == pytest.approx(sp_softmax([0.0, 1.0, 2.0]).max(), rel=1e-13)


def test_prop1_confidence_bounds_margin():
    """Proposition 1: if c > 1/2 then gamma >= log(c / (1 - c))."""
    rng = np.random.default_rng(0)
    checked = 0
    for _ in range(2000):
        V = int(rng.integers(2, 50))
        l = rng.normal(0, 1, V) * rng.uniform(0.5, 6)
        _, c = decode.top1_confidence(l[None])
        if c[0] > 0.5:
            checked += 1
            # V = 2 is the equality case; 1 - c cancels near c = 1, hence a relative slack
            bound = theory.confidence_margin_lower_bound(c[0])
            assert theory.margin(l) >= bound - 1e-9 * max(1.0, abs(bound)) - 1e-12 / (1 - c[0])
    assert checked > 100


def test_prop1_margin_condition_preserves_argmax_and_is_tight():
    rng = np.random.default_rng(1)
    for _ in range(2000):
        V = int(rng.integers(2, 40))
        l = rng.normal(0, 2, V)
        gam = theory.margin(l)
        if gam <= 0:
            continue
        d = rng.uniform(-1, 1, V)
        d *= rng.uniform(0, 0.999) * (gam / 2) / np.max(np.abs(d))
        assert theory.margin_condition_holds(l + d, l)
        assert np.argmax(l + d) == np.argmax(l)
    # tightness of the factor 2: a perturbation of exactly gamma/2 + eps can flip it
    l = np.array([1.0, 0.0, -3.0])
    gam = theory.margin(l)
    eps = 1e-6
    d = np.array([-(gam / 2 + eps), gam / 2 + eps, 0.0])
    assert not theory.margin_condition_holds(l + d, l)
    assert np.argmax(l + d) == 1


def test_g_of_delta_p_matches_paper(golden_dir):
    with open(os.path.join(golden_dir, "g_delta_p.json")) as f:
        gold = json.load(f)
    assert abs(theory.g(gold["delta_p"]) - gold["g"]) <= gold["abs_tol"]
    assert theory.g(0.5) == 0.0


def test_disagreement_losses_and_ratio():
    Y = np.array([5, 6, 7, 8])
    assert theory.accepted_disagreement([], [], Y) == 0.0
    assert theory.accepted_disagreement([0, 2], [5, 1], Y) == 0.5
    # one of three accepted tokens differs: 1/3, which no count of agreements gives
    assert theory.accepted_disagreement([0, 1, 2], [5, 6, 1], Y) == pytest.approx(1 / 3)
    assert theory.output_disagreement([5, 6, 0, 0], Y) == 0.5
    assert theory.step_ratio([3, 4], [32, 32]) == pytest.approx(7 / 64)
