"""Workload shapes and the weight-tensor numbering of the counter generator.

The tensor ids are part of the generator's definition: element ``e`` (row-major
``[out, in]``) of tensor ``t`` under seed ``s`` is a pure function of
``(s, t, e)``.  Norm weights are all ones and are not drawn.
"""
from dataclasses import dataclass

TENSOR_EMBED = 1      # [V, d]
TENSOR_LM_HEAD = 2    # [V, d]

# per-layer tensor slots; id = 100 + 16 * layer + slot
LAYER_TENSORS = {
    "wq": 0,   # [H * hd, d]
    "wk": 1,   # [Hkv * hd, d]
    "wv": 2,   # [Hkv * hd, d]
    "wo": 3,   # [d, H * hd]
    "wg": 4,   # [F, d]
    "wu": 5,   # [F, d]
    "wd": 6,   # [d, F]
    "bq": 7,   # [H * hd]      (only when qkv_bias)
    "bk": 8,   # [Hkv * hd]
    "bv": 9,   # [Hkv * hd]
}


def layer_tensor_id(layer: int, name: str) -> int:
    return 100 + 16 * layer + LAYER_TENSORS[name]


@dataclass(frozen=True)
class ModelSpec:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    mask_id: int
    qkv_bias: bool
    rms_eps: float
    rope_theta: float
    logit_scale: float
    init_std: float = 0.02

    def shapes(self, layer_name: str):
        d, H, Hkv, hd, F = self.d_model, self.n_heads, self.n_kv_heads, self.head_dim, self.ffn_dim
        return {
            "wq": (H * hd, d), "wk": (Hkv * hd, d), "wv": (Hkv * hd, d),
            "wo": (d, H * hd), "wg": (F, d), "wu": (F, d), "wd": (d, F),
            "bq": (H * hd,), "bk": (Hkv * hd,), "bv": (Hkv * hd,),
        }[layer_name]

    def with_layers(self, n_layers: int) -> "ModelSpec":
        return ModelSpec(**{**self.__dict__, "n_layers": n_layers,
                            "name": f"{self.name}-{n_layers}L"})


# Tiny masked-diffusion LM: 2 layers, d 256, 4 heads x 64, SwiGLU 688,
# eps 1e-5, theta 1e4, vocab 2048 (mask 2047), logits x8.
TINY = ModelSpec("tiny", 2, 256, 4, 4, 64, 688, 2048, 2047, False, 1e-5, 1e4, 8.0)

# LLaDA-8B shape: 32 layers, d 4096, 32 x 128 MHA, SwiGLU 12288, theta 5e5,
# vocab 126464, mask id 126336.
LLADA_8B = ModelSpec("llada8b", 32, 4096, 32, 32, 128, 12288, 126464, 126336, False,
                     1e-5, 5e5, 1.0)

# Dream-7B (Qwen2.5-7B-like) shape: 28 layers, d 3584, 28 q / 4 kv heads x 128,
# SwiGLU 18944, theta 1e6, eps 1e-6, QKV bias, vocab 152064.
DREAM_7B = ModelSpec("dream7b", 28, 3584, 28, 4, 128, 18944, 152064, 151666, True,
                     1e-6, 1e6, 1.0)
