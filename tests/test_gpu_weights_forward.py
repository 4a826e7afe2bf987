"""GPU parity: seeded weights (bit-exact) and the dense forward pass (logit tolerance).

Oracle: seeded_inputs' host generator for the weights, oracle.forward (fp64) for logits.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

import seeded_inputs as si
from oracle import forward as of
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import bf16_to_f32, logit_tolerance

pytestmark = pytest.mark.gpu

MINI_GQA = si.ModelSpec("mini-gqa", 2, 256, 4, 2, 64, 300, 1000, 999, True, 1e-6, 1e6, 6.0)
MINI_HD128 = si.ModelSpec("mini-hd128", 1, 256, 2, 1, 128, 512, 777, 5, True, 1e-6, 1e6, 6.0)
# wide enough (K >= 1024) that the QKV, output and down projections split K: partial
# workspace + the QKV finish and residual/norm kernels instead of whole-K epilogues
MID_SPLIT = si.ModelSpec("mid-split", 2, 1024, 8, 2, 128, 2816, 1000, 999, True, 1e-6, 1e6, 6.0)


def _tensors(spec):
    yield si.TENSOR_EMBED, (spec.vocab, spec.d_model)
    yield si.TENSOR_LM_HEAD, (spec.vocab, spec.d_model)
    names = ["wq", "wk", "wv", "wo", "wg", "wu", "wd"] + (["bq", "bk", "bv"] if spec.qkv_bias else [])
    for l in range(spec.n_layers):
        for n in names:
            yield si.layer_tensor_id(l, n), spec.shapes(n)


@pytest.mark.parametrize("spec", [si.TINY, MINI_GQA, MINI_HD128], ids=lambda s: s.name)
def test_weights_bit_exact(spec):
    require_gpu()
    from paper_2608_11235_amd import Model
    log_case(f"weights {spec.name}")
    with Model(spec, seed=0, max_batch=1, max_seq=64) as m:
        for tid, shape in _tensors(spec):
            n = int(np.prod(shape))
            got = m.copy_tensor(tid, n)
            want = si.gen_tensor(0, tid, shape, spec.init_std, as_bits=True).reshape(-1)
            assert (got == want).all(), f"tensor {tid}: {(got != want).sum()} mismatches"


def _check_logits(spec, B, L, row_begin, n_rows, seed=0, tag=""):
    from paper_2608_11235_amd import Model
    log_case(f"forward {spec.name} B={B} L={L} rows=[{row_begin},{row_begin + n_rows}) {tag}")
    tokens = si.prompt_tokens(seed + 1, B, L, spec.vocab, spec.mask_id)
    tokens[:, L // 2:] = spec.mask_id                    # a masked tail, as in decoding
    with Model(spec, seed=seed, max_batch=B, max_seq=L) as m:
        got = bf16_to_f32(m.forward_logits(to_dev(tokens), row_begin, n_rows).cpu().numpy())
        torch.cuda.synchronize()
    w = si.HostWeights(spec, seed)
    ref = of.forward_logits(w, spec, tokens, np.arange(row_begin, row_begin + n_rows))
    tol = logit_tolerance(ref)
    err = np.abs(got.astype(np.float64) - ref)
    rel_rms = np.sqrt(np.mean(err ** 2) / np.mean(ref ** 2))
    print(f"max_err={err.max():.4g} tol={tol:.4g} rel_rms={rel_rms:.3g}")
    assert err.max() <= tol
    return err, ref


@pytest.mark.parametrize("n_rows", [1, 20, 32, 33, 70])
def test_lm_head_only(n_rows):
    """0 layers: embedding -> final RMSNorm -> LM head: the few-row kernel at B * n_rows <= 64
    (both of its row-block widths), the tiled GEMM above, and a ragged vocab tail."""
    require_gpu()
    spec = si.ModelSpec("lmhead", 0, 192, 3, 3, 64, 64, 1000, 7, False, 1e-5, 1e4, 4.0)
    _check_logits(spec, 2, 80, 3, n_rows)


@pytest.mark.parametrize("B,L,row_begin,n_rows", [(1, 96, 32, 32), (1, 96, 0, 96), (2, 37, 5, 30),
                                                  (3, 130, 64, 64), (16, 512, 250, 40)])
def test_tiny_forward(B, L, row_begin, n_rows):
    """Small grids take the key-split attention (two wavefront groups per query tile);
    B = 16, L = 512 has 512 query-tile workgroups and takes the unsplit one."""
    require_gpu()
    _check_logits(si.TINY, B, L, row_begin, n_rows)


@pytest.mark.parametrize("spec", [MINI_GQA, MINI_HD128], ids=lambda s: s.name)
def test_gqa_bias_forward(spec):
    require_gpu()
    _check_logits(spec, 2, 100, 10, 40)


@pytest.mark.parametrize("B,L,row_begin,n_rows", [(1, 40, 0, 40), (3, 200, 150, 50), (64, 300, 100, 40)])
def test_hd128_attention_paths(B, L, row_begin, n_rows):
    """hd 128 attention, the direct-to-LDS kernel: L = 40 is one key tile, so the second
    key-range part of the small-grid launch has no tile and merges an empty state; L = 200
    splits 4 tiles over two parts, the last one partial; B = 64, L = 300 has 640 query-tile
    workgroups and takes the one-part launch, again with a partial last tile."""
    require_gpu()
    _check_logits(MINI_HD128, B, L, row_begin, n_rows)


@pytest.mark.parametrize("B,L,row_begin,n_rows", [(2, 130, 60, 40), (1, 256, 128, 32)])
def test_split_k_forward(B, L, row_begin, n_rows):
    """L = 130: row groups of 4 straddle two sequences (per-row v path); L = 256: vector v."""
    require_gpu()
    _check_logits(MID_SPLIT, B, L, row_begin, n_rows)


@pytest.mark.parametrize("spec,L", [(si.TINY, 96), (MID_SPLIT, 256)], ids=lambda v: getattr(v, "name", str(v)))
def test_forward_deterministic(spec, L):
    """Bitwise repeatable, also through the split-K partials (folded in split order)."""
    require_gpu()
    from paper_2608_11235_amd import Model
    tokens = to_dev(si.prompt_tokens(3, 2, L, spec.vocab, spec.mask_id))
    with Model(spec, seed=0, max_batch=2, max_seq=L) as m:
        runs = [m.forward_logits(tokens, 0, L).clone() for _ in range(4)]
    for r in runs[1:]:
        assert torch.equal(runs[0], r)
