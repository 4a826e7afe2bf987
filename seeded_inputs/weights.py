"""Host side of the counter-based weight generator (definition in ``wgen.c``)."""
import ctypes
import os
import subprocess

import numpy as np

from .spec import ModelSpec, TENSOR_EMBED, TENSOR_LM_HEAD, layer_tensor_id

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wgen.c")
_LIB = os.path.join(_HERE, "libwgen.so")
_lib = None


def build_wgen(force: bool = False) -> str:
    """Compile the host generator with gcc (OpenMP)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", _SRC,
                               "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build_wgen()
        lib = ctypes.CDLL(_LIB)
        lib.sgen_normal_bf16.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                         ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p]
        lib.sgen_splitmix64_stream.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p]
        lib.sgen_normal_bf16_rows.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                              ctypes.c_int64, ctypes.c_uint64, ctypes.c_double,
                                              ctypes.c_void_p]
        _lib = lib
    return _lib


def splitmix64_stream(state: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.uint64)
    _load().sgen_splitmix64_stream(state, count, out.ctypes.data)
    return out


def gen_elements(seed: int, tensor_id: int, start: int, count: int, std: float) -> np.ndarray:
    """bf16 bit patterns (uint16) of elements [start, start+count) of a tensor."""
    out = np.empty(count, dtype=np.uint16)
    if count:
        _load().sgen_normal_bf16(seed, tensor_id, start, count, std, out.ctypes.data)
    return out


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def gen_tensor(seed: int, tensor_id: int, shape, std: float = 0.02, as_bits=False):
    n = int(np.prod(shape))
    bits = gen_elements(seed, tensor_id, 0, n, std).reshape(shape)
    return bits if as_bits else bf16_bits_to_f32(bits)


def gen_rows(seed: int, tensor_id: int, rows, row_len: int, std: float = 0.02):
    """Selected rows of a row-major [*, row_len] tensor, as float32 values."""
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    out = np.empty((rows.size, row_len), dtype=np.uint16)
    if rows.size:
        _load().sgen_normal_bf16_rows(seed, tensor_id, rows.ctypes.data, rows.size, row_len,
                                      std, out.ctypes.data)
    return bf16_bits_to_f32(out)


def gen_layer(spec: ModelSpec, seed: int, layer: int) -> dict:
    """All weights of one layer as float32 arrays holding bf16 values, logical [out, in]."""
    names = ["wq", "wk", "wv", "wo", "wg", "wu", "wd"]
    if spec.qkv_bias:
        names += ["bq", "bk", "bv"]
    w = {n: gen_tensor(seed, layer_tensor_id(layer, n), spec.shapes(n), spec.init_std)
         for n in names}
    for n in ("attn_norm", "mlp_norm"):
        w[n] = np.ones(spec.d_model, dtype=np.float32)
    return w


class HostWeights:
    """Lazily generated host copy of a model's weights (float32 holding bf16 values).

    Layers are produced on demand so that full-width models can be streamed
    layer by layer; the embedding is generated only for the rows asked for.
    """

    def __init__(self, spec: ModelSpec, seed: int, cache_layers: bool = True):
        self.spec, self.seed, self.cache_layers = spec, seed, cache_layers
        self._layers = {}
        self._lm_head = None
        self.final_norm = np.ones(spec.d_model, dtype=np.float32)

    def embed_rows(self, token_ids) -> np.ndarray:
        return gen_rows(self.seed, TENSOR_EMBED, token_ids, self.spec.d_model, self.spec.init_std)

    def layer(self, i: int) -> dict:
        if i in self._layers:
            return self._layers[i]
        w = gen_layer(self.spec, self.seed, i)
        if self.cache_layers:
            self._layers[i] = w
        return w

    def lm_head(self) -> np.ndarray:
        if self._lm_head is None:
            self._lm_head = gen_tensor(self.seed, TENSOR_LM_HEAD,
                                       (self.spec.vocab, self.spec.d_model), self.spec.init_std)
        return self._lm_head
