"""The Python binding refuses tensors the C ABI would misread, before any library call:
host tensors and non-tensors here on the CPU (the GPU-side dtype, contiguity and size
refusals are in the GPU hook tests)."""
import numpy as np
import pytest
import torch

import seeded_inputs as si
from paper_2608_11235_amd import api


def test_host_tensor_and_non_tensor_refused():
    with pytest.raises(ValueError, match="GPU"):
        api.check_device_tensor(torch.zeros(4, dtype=torch.int32), "t", (torch.int32,))
    with pytest.raises(TypeError):
        api.check_device_tensor(np.zeros(4, np.int32), "t", (torch.int32,))


def test_model_calls_check_before_the_library():
    m = api.Model.__new__(api.Model)   # no library handle: a check must fail first
    m.spec = si.TINY
    with pytest.raises(ValueError, match="tokens"):
        m.forward_logits(torch.zeros((1, 8), dtype=torch.int32), 0, 1)
    with pytest.raises(ValueError, match="prompt"):
        m.block_decode(torch.zeros((1, 8), dtype=torch.int32), 32, api.Sched(16, 4), api.Gate())


def test_host_state_refused():
    st = api.DecodeState(1, 8, 32, 16, 16, device="cpu")
    with pytest.raises(ValueError, match="state.tokens"):
        st.c()
