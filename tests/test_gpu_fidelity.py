"""Fidelity harness (NEXT item): dense vs CORA decodes on the GPU, their step ratio and the
disagreement metrics L^acc (Eq. 7, per prompt, averaged over the prompts) and L^out
(Eq. 12) against the dense endpoint.

The harness (bench.fidelity_run) computes the metrics from the GPU decodes itself; here the
oracle's definitions (oracle.theory, pinned in test_oracle_scores) are applied to the same
decodes and must give the same numbers, and the harness's structural facts are checked:
the dense decode runs the full horizon, the gate never adds passes, the replay that records
acceptances reproduces the timed decode, and with the gate off nothing is accepted.
"""
from dataclasses import replace

import numpy as np
import pytest

import seeded_inputs as si
from oracle import theory
from tests.gpu_common import log_case, require_gpu

pytestmark = pytest.mark.gpu

SPEC = replace(si.TINY, name="tiny-std0.07", init_std=0.07, logit_scale=2.0)
P, G, BLK, S = 32, 64, 32, 16


def _run(delta_p, m_req, scope, gate_enabled=True):
    import bench
    from paper_2608_11235_amd import Model
    prompt = si.prompt_tokens(1, 2, P, SPEC.vocab, SPEC.mask_id)
    with Model(SPEC, seed=0, max_batch=2, max_seq=P + G) as m:
        if gate_enabled:
            return bench.fidelity_run(m, prompt, G, BLK, S, delta_p, m_req, scope)
        return bench.fidelity_run(m, prompt, G, BLK, S, 2.0, m_req, scope)  # c <= 1 < 2


@pytest.mark.parametrize("scope", [0, 1])
@pytest.mark.parametrize("delta_p,m_req", [(0.05, 1), (0.02, 0), (0.1, 2)])
def test_fidelity_metrics_follow_their_definitions(delta_p, m_req, scope):
    require_gpu()
    log_case(f"fidelity dp={delta_p} m={m_req} scope={scope}")
    r = _run(delta_p, m_req, scope)
    a, c = r["arrays"], r["cora"]
    y_d, y = a["dense_tokens"], a["cora_tokens"]
    assert (a["dense_passes"] == S).all()                      # dense horizon
    assert (a["cora_passes"] <= a["dense_passes"]).all()        # the gate never adds passes
    assert c["replay_matches_block_decode"]
    assert c["rho"] == pytest.approx(theory.step_ratio(a["cora_passes"], a["dense_passes"]),
                                     abs=5e-5)
    assert c["L_out"] == pytest.approx(theory.output_disagreement(y[:, P:], y_d[:, P:]))
    # Eq. (7) per prompt (0 when the gate accepted nothing), averaged over the prompts
    n, per_prompt = 0, []
    for b, acc in enumerate(a["accepted"]):
        pos, tok = (list(x) for x in zip(*acc)) if acc else ([], [])
        per_prompt.append(theory.accepted_disagreement(pos, tok, y_d[b]))
        n += len(acc)
        assert all(y[b, i] == t for i, t in acc)               # accepted tokens stay committed
    assert c["accepted"] == n
    assert c["L_acc"] == pytest.approx(float(np.mean(per_prompt)))
    print(f"rho {c['rho']}, accepted {n}, L_acc {c['L_acc']:.3f}, L_out {c['L_out']:.3f}")
    assert n > 0, "the gate should fire at this threshold"


def test_fidelity_gate_unreachable_is_dense():
    """A threshold no confidence reaches: nothing accepted, the decode is the dense one."""
    require_gpu()
    r = _run(None, 1, 0, gate_enabled=False)
    c = r["cora"]
    assert c["accepted"] == 0 and c["L_acc"] == 0.0 and c["L_out"] == 0.0 and c["rho"] == 1.0
