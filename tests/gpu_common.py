"""Shared set-up for GPU tests: skip cleanly without a GPU, fail loudly without the library."""
import os

import numpy as np
import pytest
import torch


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2608_11235_amd._lib as L
    if not os.path.exists(L.LIB_PATH):
        raise RuntimeError("GPU present but libcora.so is not built")
    return torch.device("cuda:0")


def to_dev(a, dtype=None, device="cuda"):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device)


def log_case(msg):
    print(f"[case] {msg}", flush=True)
