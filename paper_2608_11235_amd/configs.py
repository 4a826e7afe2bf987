"""Backbone shapes the library is exercised on (LLaDA-8B and Dream-7B layouts, plus a tiny one)."""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class ModelConfig:
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

    def with_layers(self, n_layers: int) -> "ModelConfig":
        return replace(self, n_layers=n_layers, name=f"{self.name}-{n_layers}L")


# 2 layers, d 256, 4 heads x 64, SwiGLU 688, vocab 2048 (mask 2047), logits x8
TINY = ModelConfig("tiny", 2, 256, 4, 4, 64, 688, 2048, 2047, False, 1e-5, 1e4, 8.0)
# LLaDA-8B layout: 32 layers, d 4096, 32 x 128 MHA, SwiGLU 12288, vocab 126464
LLADA_8B = ModelConfig("llada8b", 32, 4096, 32, 32, 128, 12288, 126464, 126336, False,
                       1e-5, 5e5, 1.0)
# Dream-7B layout: 28 layers, d 3584, 28 q / 4 kv heads x 128, SwiGLU 18944, QKV bias
DREAM_7B = ModelConfig("dream7b", 28, 3584, 28, 4, 128, 18944, 152064, 151666, True,
                       1e-6, 1e6, 1.0)
