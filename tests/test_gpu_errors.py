"""Error paths that need a device: allocation failure at create, and the argument checks of
the calls that take a model.  Every case fails in host code before any kernel runs, and
the device stays usable afterwards."""
import numpy as np
import pytest
import torch

import seeded_inputs as si
from tests.gpu_common import log_case, require_gpu, to_dev

pytestmark = pytest.mark.gpu


def _tiny_forward_works():
    from paper_2608_11235_amd import Model
    tokens = to_dev(si.prompt_tokens(2, 1, 64, si.TINY.vocab, si.TINY.mask_id))
    with Model(si.TINY, seed=0, max_batch=1, max_seq=64) as m:
        lg = m.forward_logits(tokens, 0, 8)
        torch.cuda.synchronize()
    assert lg.shape == (1, 8, si.TINY.vocab)


def test_create_out_of_memory():
    """LLaDA-8B width with 1000 layers needs ~436 GB of weights: the allocation fails and
    create reports CORA_ERR_OOM with the HIP message; nothing is left allocated."""
    require_gpu()
    from paper_2608_11235_amd import LLADA_8B, Model
    from paper_2608_11235_amd._lib import CoraError
    log_case("create 1000-layer LLaDA width (expect OOM)")
    free0, _ = torch.cuda.mem_get_info()
    with pytest.raises(CoraError) as ei:
        Model(LLADA_8B.with_layers(1000), seed=0, max_batch=1, max_seq=64)
    assert ei.value.status == -3
    assert "allocation" in str(ei.value)
    free1, _ = torch.cuda.mem_get_info()
    assert free1 >= free0 - (64 << 20)
    _tiny_forward_works()


def test_calls_reject_arguments_outside_the_model():
    require_gpu()
    from paper_2608_11235_amd import DecodeState, Gate, Model, Sched
    from paper_2608_11235_amd._lib import CoraError
    log_case("argument checks of forward_logits / denoise_step / block_decode")
    spec, P, G = si.TINY, 32, 64
    with Model(spec, seed=0, max_batch=2, max_seq=P + G) as m:
        tokens = to_dev(si.prompt_tokens(4, 2, P + G, spec.vocab, spec.mask_id))
        with pytest.raises(CoraError) as ei:       # rows past the canvas
            m.forward_logits(tokens, P + G - 4, 8)
        assert ei.value.status == -1
        big = to_dev(si.prompt_tokens(4, 3, P + G, spec.vocab, spec.mask_id))
        with pytest.raises(CoraError) as ei:       # batch beyond max_batch
            m.forward_logits(big, 0, 8)
        assert ei.value.status == -1
        host = si.initial_decode_state(si.prompt_tokens(5, 3, P, spec.vocab, spec.mask_id), G,
                                       spec.mask_id)
        st = DecodeState.from_host(host, P, G, 32, 32)
        with pytest.raises(CoraError) as ei:       # state batch beyond max_batch
            m.denoise_step(st, Sched(32, 8), Gate(0.65, 1, True))
        assert ei.value.status == -1
        host = si.initial_decode_state(si.prompt_tokens(5, 1, P, spec.vocab, spec.mask_id), G,
                                       spec.mask_id)
        st = DecodeState.from_host(host, P, G, 32, 32)
        with pytest.raises(CoraError) as ei:       # steps_per_block > block_len
            m.denoise_step(st, Sched(32, 33), Gate(0.65, 1, True))
        assert ei.value.status == -1
        prompt = to_dev(si.prompt_tokens(6, 1, P, spec.vocab, spec.mask_id))
        with pytest.raises(CoraError) as ei:       # gen_len not a multiple of block_len
            m.block_decode(prompt, 48, Sched(32, 8), Gate(0.65, 1, True))
        assert ei.value.status in (-1, -2)
        # the model still decodes after the refused calls
        y, passes, total = m.block_decode(prompt, G, Sched(32, 8), Gate(0.65, 1, True))
        assert y.shape == (1, P + G) and int(total) >= 1
        assert (y[:, P:] != spec.mask_id).all()
