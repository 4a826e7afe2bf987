"""Pythonic wrappers over the C ABI (marshalling only)."""
import ctypes
from typing import Optional
from dataclasses import dataclass

import numpy as np
import torch

from . import _lib
from ._lib import check, ptr, stream_handle

TENSOR_EMBED = 1
TENSOR_LM_HEAD = 2
_LAYER_SLOTS = {"wq": 0, "wk": 1, "wv": 2, "wo": 3, "wg": 4, "wu": 5, "wd": 6,
                "bq": 7, "bk": 8, "bv": 9}


_BF16_BITS = (torch.int16, torch.bfloat16, torch.uint16)


def check_device_tensor(t, name, dtypes, numel=None):
    """Refuse what the C ABI would misread: a host or non-contiguous tensor, another element
    type, or fewer elements than the call reads or writes (the library sees only a pointer)."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: must be a GPU tensor (got device {t.device})")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, the call needs {numel}")
    return t


def layer_tensor_id(layer: int, name: str) -> int:
    return 100 + 16 * layer + _LAYER_SLOTS[name]


def model_cfg_from(spec) -> _lib.ModelCfg:
    """Build the C struct from any object carrying the backbone fields."""
    return _lib.ModelCfg(spec.n_layers, spec.d_model, spec.n_heads, spec.n_kv_heads,
                         spec.head_dim, spec.ffn_dim, spec.vocab, spec.mask_id,
                         int(bool(spec.qkv_bias)), spec.rms_eps, spec.rope_theta,
                         spec.logit_scale, float(getattr(spec, "init_std", 0.02)))


@dataclass
class Sched:
    block_len: int = 32
    steps_per_block: int = 32
    eos_id: Optional[int] = None   # EOS-aware controller when set

    def c(self):
        return _lib.SchedCfg(self.block_len, self.steps_per_block,
                             0 if self.eos_id is None else 1,
                             0 if self.eos_id is None else int(self.eos_id))


@dataclass
class Gate:
    delta_p: float = 0.65
    m_req: int = 1
    enabled: bool = True
    persist_scope: int = 0

    def c(self):
        return _lib.GateCfg(self.delta_p, self.m_req, int(self.enabled), self.persist_scope)


class DecodeState:
    """Device-resident decode state (see cora_state in include/cora.h)."""

    def __init__(self, B, prompt_len, gen_len, n_rows, block_len, device="cuda", passes=True):
        i32, u8 = torch.int32, torch.uint8
        L = prompt_len + gen_len
        self.B, self.prompt_len, self.gen_len, self.block_len = B, prompt_len, gen_len, block_len
        self.tokens = torch.zeros((B, L), dtype=i32, device=device)
        self.unresolved = torch.zeros((B, L), dtype=u8, device=device)
        self.prev_top1 = torch.full((B, L), -1, dtype=i32, device=device)
        self.persist = torch.zeros((B, L), dtype=i32, device=device)
        self.block_idx = torch.zeros(B, dtype=i32, device=device)
        self.step_idx = torch.zeros(B, dtype=i32, device=device)
        self.top1 = torch.zeros((B, n_rows), dtype=i32, device=device)
        self.conf = torch.zeros((B, n_rows), dtype=torch.float32, device=device)
        self.decision = torch.zeros((B, block_len), dtype=u8, device=device)
        self.done = torch.zeros(B, dtype=i32, device=device)
        n_blocks = gen_len // block_len
        self.passes = torch.zeros((B, n_blocks), dtype=i32, device=device) if passes else None

    @classmethod
    def from_host(cls, host: dict, prompt_len, gen_len, n_rows, block_len, device="cuda"):
        """Copy a host state dict (numpy arrays as in seeded_inputs) to the device."""
        B = host["tokens"].shape[0]
        st = cls(B, prompt_len, gen_len, n_rows, block_len, device)
        st.load(host)
        return st

    def load(self, host: dict):
        for name in ("tokens", "unresolved", "prev_top1", "persist", "block_idx", "step_idx"):
            src = torch.from_numpy(np.ascontiguousarray(host[name]))
            getattr(self, name).copy_(src.to(getattr(self, name).dtype))

    def to_host(self) -> dict:
        names = ("tokens", "unresolved", "prev_top1", "persist", "block_idx", "step_idx", "top1",
                 "conf", "decision", "done")
        out = {n: getattr(self, n).cpu().numpy() for n in names}
        if self.passes is not None:
            out["passes"] = self.passes.cpu().numpy()
        return out

    def c(self):
        B, L = self.B, self.prompt_len + self.gen_len
        for name, dt, n in (("tokens", torch.int32, B * L), ("unresolved", torch.uint8, B * L),
                            ("prev_top1", torch.int32, B * L), ("persist", torch.int32, B * L),
                            ("block_idx", torch.int32, B), ("step_idx", torch.int32, B),
                            ("top1", torch.int32, None), ("conf", torch.float32, None),
                            ("decision", torch.uint8, None), ("done", torch.int32, B)):
            check_device_tensor(getattr(self, name), f"state.{name}", (dt,), n)
        if self.passes is not None:
            check_device_tensor(self.passes, "state.passes", (torch.int32,),
                                B * (self.gen_len // self.block_len))
        return _lib.State(ptr(self.tokens), ptr(self.unresolved), ptr(self.prev_top1),
                          ptr(self.persist), ptr(self.block_idx), ptr(self.step_idx),
                          ptr(self.top1), ptr(self.conf), ptr(self.decision), ptr(self.done),
                          ptr(self.passes), self.B, self.prompt_len, self.gen_len)


class Model:
    """Seeded backbone + workspace owned by libcora (weights drawn on the GPU)."""

    def __init__(self, spec, seed: int, max_batch: int, max_seq: int, stream=None):
        lib = _lib.load()
        self.spec, self.seed, self.max_batch, self.max_seq = spec, seed, max_batch, max_seq
        self._cfg = model_cfg_from(spec)
        h = ctypes.c_void_p()
        check(lib.cora_model_create(ctypes.byref(self._cfg), seed, max_batch, max_seq,
                                    stream_handle(stream), ctypes.byref(h)), "cora_model_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None) and self._h.value:
            _lib.load().cora_model_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @property
    def handle(self):
        return self._h

    def forward_logits(self, tokens, row_begin, n_rows, out=None, stream=None):
        check_device_tensor(tokens, "tokens", (torch.int32,))
        B, L = tokens.shape
        if out is None:
            out = torch.empty((B, n_rows, self.spec.vocab), dtype=torch.int16,
                              device=tokens.device)
        check_device_tensor(out, "out", _BF16_BITS, B * n_rows * self.spec.vocab)
        check(_lib.load().cora_forward_logits(self._h, ptr(tokens), B, L, row_begin, n_rows,
                                               ptr(out), stream_handle(stream)),
              "cora_forward_logits")
        return out

    def denoise_step(self, state: DecodeState, sched: Sched, gate: Gate, stream=None):
        st, sc, gt = state.c(), sched.c(), gate.c()
        check(_lib.load().cora_denoise_step(self._h, ctypes.byref(st), ctypes.byref(sc),
                                             ctypes.byref(gt), stream_handle(stream)),
              "cora_denoise_step")

    def block_decode(self, prompt, gen_len, sched: Sched, gate: Gate, out=None, stream=None):
        check_device_tensor(prompt, "prompt", (torch.int32,))
        B, P = prompt.shape
        if out is None:
            out = torch.empty((B, P + gen_len), dtype=torch.int32, device=prompt.device)
        check_device_tensor(out, "out", (torch.int32,), B * (P + gen_len))
        n_blocks = gen_len // sched.block_len
        passes = np.zeros((B, n_blocks), dtype=np.int32)
        total = ctypes.c_int32(0)
        sc, gt = sched.c(), gate.c()
        check(_lib.load().cora_block_decode(self._h, ptr(prompt), B, P, gen_len, ctypes.byref(sc),
                                             ctypes.byref(gt), ptr(out),
                                             ctypes.c_void_p(passes.ctypes.data),
                                             ctypes.byref(total), stream_handle(stream)),
              "cora_block_decode")
        return out, passes, int(total.value)

    def copy_tensor(self, tensor_id: int, n_elements: int) -> np.ndarray:
        out = np.empty(n_elements, dtype=np.uint16)
        check(_lib.load().cora_model_copy_tensor(self._h, tensor_id,
                                                  ctypes.c_void_p(out.ctypes.data), out.nbytes),
              "cora_model_copy_tensor")
        return out

    def set_compaction(self, enable: bool):
        check(_lib.load().cora_model_set_compaction(self._h, int(enable)),
              "cora_model_set_compaction")

    def set_timing(self, enable: bool):
        check(_lib.load().cora_model_set_timing(self._h, int(enable)), "cora_model_set_timing")

    def read_timing(self):
        ms, n = ctypes.c_double(0), ctypes.c_int64(0)
        check(_lib.load().cora_model_read_timing(self._h, ctypes.byref(ms), ctypes.byref(n)),
              "cora_model_read_timing")
        return ms.value, n.value

    def device_bytes(self):
        w, ws = ctypes.c_size_t(0), ctypes.c_size_t(0)
        check(_lib.load().cora_model_device_bytes(self._h, ctypes.byref(w), ctypes.byref(ws)),
              "cora_model_device_bytes")
        return w.value, ws.value


def vocab_gate(logits, n_rows, row_begin, V, mask_id, state: DecodeState, k_transfer,
               sched: Sched, gate: Gate, stream=None):
    check_device_tensor(logits, "logits", _BF16_BITS, state.B * n_rows * V)
    st, sc, gt = state.c(), sched.c(), gate.c()
    check(_lib.load().cora_vocab_gate(ptr(logits), n_rows, row_begin, V, mask_id,
                                       ctypes.byref(st), k_transfer, ctypes.byref(sc),
                                       ctypes.byref(gt), stream_handle(stream)),
          "cora_vocab_gate")


def vocab_gate_noalloc(logits, n_rows, row_begin, V, mask_id, state: DecodeState, k_transfer,
                       sched: Sched, gate: Gate, stream=None):
    """cora_vocab_gate_noalloc: vocab_gate without any allocation (split rows, fixed scratch)."""
    check_device_tensor(logits, "logits", _BF16_BITS, state.B * n_rows * V)
    st, sc, gt = state.c(), sched.c(), gate.c()
    check(_lib.load().cora_vocab_gate_noalloc(ptr(logits), n_rows, row_begin, V, mask_id,
                                               ctypes.byref(st), k_transfer, ctypes.byref(sc),
                                               ctypes.byref(gt), stream_handle(stream)),
          "cora_vocab_gate_noalloc")
