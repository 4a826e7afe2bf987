"""Host-side arithmetic of bench.py (CPU only).

The roofline figures divide by algorithmic FLOPs; these are pinned to the per-pass totals
worked out separately from the model shapes (GEMMs 2·M·N·K, attention 4·B·H·L²·hd, LM
head 2·rows·d·V on the scored rows): 7.317 TFLOP for LLaDA-8B at B 1, L 512 with 32
scored rows; 54.576 TFLOP for Dream-7B at B 8, L 512 with 8 x 32 rows; 18.759 TFLOP for
LLaDA-8B at L 1280; 103.08 GFLOP for one gate/up launch at M 512.  Also: counter traffic
is withheld once the kernel source no longer matches the digest the counters were taken
on, and more than one GPU is refused before anything touches a device."""
import os
import subprocess
import sys

import pytest

import bench
import seeded_inputs as si

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("spec,M,rows,batch,tflop", [
    (si.LLADA_8B, 512, 32, 1, 7.317),
    (si.DREAM_7B, 8 * 512, 8 * 32, 8, 54.576),
    (si.LLADA_8B, 1280, 32, 1, 18.759),
])
def test_pass_flops_match_the_shape_totals(spec, M, rows, batch, tflop):
    assert bench.pass_flops(spec, M, rows, batch=batch) / 1e12 == pytest.approx(tflop, abs=6e-4)


def test_gate_up_flops():
    assert bench.gu_flops(si.LLADA_8B, 512) / 1e9 == pytest.approx(103.08, abs=6e-3)


def test_attention_share_is_quadratic_in_length():
    # attention is the only term that grows faster than M: with the LM head fixed,
    # f(2L) - 2 f(L) = layers x 4 H hd (4 L^2 - 2 L^2) = twice the attention FLOPs at L
    spec = si.LLADA_8B
    lm = 2 * 32 * spec.d_model * spec.vocab
    f1 = bench.pass_flops(spec, 512, 32) - lm
    f2 = bench.pass_flops(spec, 1024, 32) - lm
    attn1 = spec.n_layers * 4 * spec.n_heads * 512 * 512 * spec.head_dim
    assert f2 - 2 * f1 == 2 * attn1


def test_counter_traffic_needs_matching_digest(monkeypatch):
    path = "paper_2608_11235_amd/csrc/vocab_gate.hip"
    digest = bench.source_digest(path)
    monkeypatch.setitem(bench.COUNTER_TRAFFIC, "probe", (path, digest, 123))
    assert bench.counter_traffic("probe") == 123
    monkeypatch.setitem(bench.COUNTER_TRAFFIC, "probe", (path, "0" * 16, 123))
    assert bench.counter_traffic("probe") is None


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""
