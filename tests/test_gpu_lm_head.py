"""GPU checks of the few-row LM head (packed weights) and of the step's fused scores.

A denoising step computes Eq. (1) inside the LM-head pass and never writes logits: with at
most 64 scored rows (B x block rows) in the packed-weight stream, with more in the tiled
GEMM's top-1 epilogue.  Two properties tie the paths together at any size:

* the fused top-1 of a row is the lowest id among the maxima of the same rounded logits
  that the logits mode of the same path writes (mask id left out), bit for bit, and its
  confidence is 1 / sum_v exp(l_v - l_max) of those logits within fp32 summation error;
* the few-row kernel's logits equal the tiled GEMM's (large-row path) up to fp32 summation
  order: at most one bf16 unit in the last place apart.

Logit parity with the oracle for both paths is in test_gpu_weights_forward.py.
"""
import numpy as np
import pytest
import torch

import seeded_inputs as si
from tests.gpu_common import log_case, require_gpu, to_dev
from tests.parity import bf16_to_f32

pytestmark = pytest.mark.gpu

# 0 layers (embedding -> final norm -> LM head), d = 192 (3 K-stages, fewer than the
# kernel's 4-deep ring), vocab 5000 (not a multiple of 32 or 128: a partial weight group
# and a partial workgroup)
RAGGED = si.ModelSpec("lmhead-ragged", 0, 192, 3, 3, 64, 64, 5000, 4321, False, 1e-5, 1e4, 3.0)
# the LLaDA-8B vocabulary and width without layers: 988 workgroups, 64 K-stages
LLADA_HEAD = si.ModelSpec("lmhead-llada", 0, 4096, 32, 32, 128, 128, 126464, 126336, False,
                          1e-5, 5e5, 1.0)
# 0 layers, vocab 24100 at 512 scored rows: the planner takes the 256 x 192 tile, whose last
# tile column holds 100 valid columns (one wavefront column range entirely past the vocab)
WIDE = si.ModelSpec("lmhead-wide", 0, 256, 4, 4, 64, 64, 24100, 24007, False, 1e-5, 1e4, 2.0)
BLK = 32


def _host_scores(logits, mask_id):
    """Lowest-id argmax and 1/sum exp(l - max) of rounded logits [..., V], mask id left out."""
    x = logits.astype(np.float64).copy()
    x[..., mask_id] = -np.inf
    top = np.argmax(x, axis=-1)                       # first occurrence of the maximum
    mx = np.take_along_axis(x, top[..., None], -1)
    conf = 1.0 / np.exp(x - mx).sum(-1)
    return top, conf


@pytest.mark.parametrize("spec,B,blk", [(si.TINY, 1, BLK), (si.TINY, 2, BLK), (si.TINY, 3, BLK),
                                        (RAGGED, 1, BLK), (RAGGED, 2, BLK), (RAGGED, 3, BLK),
                                        (WIDE, 2, 256)],
                         ids=lambda v: getattr(v, "name", str(v)))
def test_fused_scores_match_own_logits(spec, B, blk):
    """B x blk = 32, 64: packed-weight stream; 96 (256 x 128 tiles), 512 (256 x 192 tiles):
    the tiled GEMM's top-1 epilogue."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    P, G = 32, max(64, blk)
    L = P + G
    log_case(f"fused scores {spec.name} B={B} blk={blk}")
    tokens = si.prompt_tokens(11, B, L, spec.vocab, spec.mask_id)
    tokens[:, P:] = spec.mask_id
    tokens[:, P + 3:P + 9] = tokens[:, 3:9]            # a few resolved positions in the block
    host = dict(tokens=tokens.astype(np.int32), unresolved=(tokens == spec.mask_id).astype(np.uint8),
                prev_top1=np.full((B, L), -1, np.int32), persist=np.zeros((B, L), np.int32),
                block_idx=np.zeros(B, np.int32), step_idx=np.zeros(B, np.int32))
    with Model(spec, seed=0, max_batch=B, max_seq=L) as m:
        lg = bf16_to_f32(m.forward_logits(to_dev(host["tokens"]), P, blk).cpu().numpy())
        st = DecodeState.from_host(host, P, G, blk, blk)
        m.denoise_step(st, Sched(blk, 8), Gate(0.65, 1, True))
        out = st.to_host()
    top, conf = _host_scores(lg, spec.mask_id)
    assert (out["top1"] == top).all(), f"{(out['top1'] != top).sum()} top-1 mismatches"
    rel = np.abs(out["conf"].astype(np.float64) - conf) / conf
    assert rel.max() <= 2e-5, f"confidence rel err {rel.max():.3g}"


@pytest.mark.parametrize("spec,B,n_rows", [(RAGGED, 1, 20), (RAGGED, 2, 32), (si.TINY, 1, 32),
                                           (LLADA_HEAD, 1, 32), (LLADA_HEAD, 2, 32)],
                         ids=lambda v: getattr(v, "name", str(v)))
def test_few_row_logits_match_tiled_gemm(spec, B, n_rows):
    """Rows [r0, r0 + n_rows) through the few-row kernel (B * n_rows <= 64) against the same
    rows inside a 96-row call (tiled GEMM)."""
    require_gpu()
    from paper_2608_11235_amd import Model
    L, r0 = 128, 40
    log_case(f"few-row logits {spec.name} B={B} rows={n_rows}")
    tokens = to_dev(si.prompt_tokens(5, B, L, spec.vocab, spec.mask_id))
    with Model(spec, seed=0, max_batch=B, max_seq=L) as m:
        few = m.forward_logits(tokens, r0, n_rows).clone()
        many = m.forward_logits(tokens, r0 - 16, 96)[:, 16:16 + n_rows].clone()
    a = bf16_to_f32(few.cpu().numpy()).astype(np.float64)
    b = bf16_to_f32(many.cpu().numpy()).astype(np.float64)
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(a), np.abs(b)) + 1e-30)) - 7)
    diff = np.abs(a - b)
    print(f"[summary] {spec.name}: words differing {(diff > 0).sum()} of {diff.size}, "
          f"max diff / ulp {np.max(diff / ulp):.2f}")
    assert (diff <= ulp).all()


@pytest.mark.parametrize("B", [1, 8])
def test_fused_scores_llada_vocab(B):
    """The fused paths at the LLaDA-8B head shape (126464 x 4096, 32-row blocks): B = 1 in
    the packed-weight stream, B = 8 (256 rows) in the tiled GEMM's top-1 epilogue."""
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    spec, P, G = LLADA_HEAD, 64, 64
    L = P + G
    log_case(f"fused scores llada head B={B}")
    tokens = si.prompt_tokens(7, B, L, spec.vocab, spec.mask_id)
    tokens[:, P:] = spec.mask_id
    tokens[:, P + 1:P + 20] = tokens[:, 1:20]
    host = dict(tokens=tokens.astype(np.int32), unresolved=(tokens == spec.mask_id).astype(np.uint8),
                prev_top1=np.full((B, L), -1, np.int32), persist=np.zeros((B, L), np.int32),
                block_idx=np.zeros(B, np.int32), step_idx=np.zeros(B, np.int32))
    with Model(spec, seed=0, max_batch=B, max_seq=L) as m:
        lg = bf16_to_f32(m.forward_logits(to_dev(host["tokens"]), P, BLK).cpu().numpy())
        st = DecodeState.from_host(host, P, G, BLK, BLK)
        m.denoise_step(st, Sched(BLK, 32), Gate(0.65, 1, True))
        torch.cuda.synchronize()
        out = st.to_host()
    top, conf = _host_scores(lg, spec.mask_id)
    assert (out["top1"] == top).all()
    rel = np.abs(out["conf"].astype(np.float64) - conf) / conf
    assert rel.max() <= 1e-4, f"confidence rel err {rel.max():.3g}"
