"""ctypes binding of libcora.so (argument marshalling only).

Every step of the denoising pass runs in the HIP library; this module only
turns torch device tensors into pointers and the current HIP stream into a
handle.  Loading fails loudly when the library has not been built.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcora.so")

c_i32, c_u64, c_f32, c_f64, c_vp, c_sz = (ctypes.c_int32, ctypes.c_uint64, ctypes.c_float,
                                          ctypes.c_double, ctypes.c_void_p, ctypes.c_size_t)


class ModelCfg(ctypes.Structure):
    _fields_ = [("n_layers", c_i32), ("d_model", c_i32), ("n_heads", c_i32),
                ("n_kv_heads", c_i32), ("head_dim", c_i32), ("ffn_dim", c_i32), ("vocab", c_i32),
                ("mask_id", c_i32), ("qkv_bias", c_i32), ("rms_eps", c_f32),
                ("rope_theta", c_f32), ("logit_scale", c_f32), ("init_std", c_f64)]


class SchedCfg(ctypes.Structure):
    _fields_ = [("block_len", c_i32), ("steps_per_block", c_i32), ("eos_enabled", c_i32),
                ("eos_id", c_i32)]


class GateCfg(ctypes.Structure):
    _fields_ = [("delta_p", c_f32), ("m_req", c_i32), ("gate_enabled", c_i32),
                ("persist_scope", c_i32)]


class State(ctypes.Structure):
    _fields_ = [("tokens", c_vp), ("unresolved", c_vp), ("prev_top1", c_vp), ("persist", c_vp),
                ("block_idx", c_vp), ("step_idx", c_vp), ("top1", c_vp), ("conf", c_vp),
                ("decision", c_vp), ("done", c_vp), ("passes", c_vp), ("B", c_i32),
                ("prompt_len", c_i32), ("gen_len", c_i32)]


EXPORTS = {
    "cora_model_create": (c_i32, [ctypes.POINTER(ModelCfg), c_u64, c_i32, c_i32, c_vp,
                                  ctypes.POINTER(c_vp)]),
    "cora_model_destroy": (c_i32, [c_vp]),
    "cora_forward_logits": (c_i32, [c_vp, c_vp, c_i32, c_i32, c_i32, c_i32, c_vp, c_vp]),
    "cora_denoise_step": (c_i32, [c_vp, ctypes.POINTER(State), ctypes.POINTER(SchedCfg),
                                  ctypes.POINTER(GateCfg), c_vp]),
    "cora_vocab_gate": (c_i32, [c_vp, c_i32, c_i32, c_i32, c_i32, ctypes.POINTER(State), c_i32,
                                ctypes.POINTER(SchedCfg), ctypes.POINTER(GateCfg), c_vp]),
    "cora_vocab_gate_noalloc": (c_i32, [c_vp, c_i32, c_i32, c_i32, c_i32, ctypes.POINTER(State),
                                        c_i32, ctypes.POINTER(SchedCfg), ctypes.POINTER(GateCfg),
                                        c_vp]),
    "cora_block_decode": (c_i32, [c_vp, c_vp, c_i32, c_i32, c_i32, ctypes.POINTER(SchedCfg),
                                  ctypes.POINTER(GateCfg), c_vp, c_vp, c_vp, c_vp]),
    "cora_model_copy_tensor": (c_i32, [c_vp, c_i32, c_vp, c_sz]),
    "cora_model_set_timing": (c_i32, [c_vp, c_i32]),
    "cora_model_set_compaction": (c_i32, [c_vp, c_i32]),
    "cora_model_read_timing": (c_i32, [c_vp, ctypes.POINTER(c_f64), ctypes.POINTER(ctypes.c_int64)]),
    "cora_model_device_bytes": (c_i32, [c_vp, ctypes.POINTER(c_sz), ctypes.POINTER(c_sz)]),
    "cora_last_error": (ctypes.c_char_p, []),
}

_lib = None


class CoraError(RuntimeError):
    def __init__(self, status, func, msg):
        super().__init__(f"{func} failed with status {status}: {msg}")
        self.status = status


def load(path: str = LIB_PATH):
    """Load libcora.so and declare every exported symbol; raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() "
                          "(python -m paper_2608_11235_amd.build)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in EXPORTS.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    _lib = lib
    return lib


def check(status, func):
    if status != 0:
        raise CoraError(status, func, load().cora_last_error().decode())


def stream_handle(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)
