"""Pins of the oracle's dense forward pass.

Against torch's CPU library routines written independently here (linear,
rms_norm, silu, scaled_dot_product_attention, RoPE as complex rotation, GQA by
repeat_interleave), plus RoPE's relative-position identity and closed-form
attention cases.  fp64 on both sides.
"""
from types import SimpleNamespace

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import forward as of


def _spec(**kw):
    base = dict(n_layers=2, d_model=32, n_heads=4, n_kv_heads=4, head_dim=8, ffn_dim=40,
                vocab=50, qkv_bias=False, rms_eps=1e-5, rope_theta=1e4, logit_scale=3.0)
    base.update(kw)
    return SimpleNamespace(**base)


class _Weights:
    def __init__(self, spec, seed):
        rng = np.random.default_rng(seed)
        d, H, Hkv, hd, F_, V = (spec.d_model, spec.n_heads, spec.n_kv_heads, spec.head_dim,
                                spec.ffn_dim, spec.vocab)
        n = lambda *s: rng.normal(0, 0.3, s)  # noqa: E731
        self.E, self.lm, self.final_norm = n(V, d), n(V, d), 1 + 0.1 * n(d)
        self.layers = []
        for _ in range(spec.n_layers):
            w = dict(wq=n(H * hd, d), wk=n(Hkv * hd, d), wv=n(Hkv * hd, d), wo=n(d, H * hd),
                     wg=n(F_, d), wu=n(F_, d), wd=n(d, F_), attn_norm=1 + 0.1 * n(d),
                     mlp_norm=1 + 0.1 * n(d))
            if spec.qkv_bias:
                w.update(bq=n(H * hd), bk=n(Hkv * hd), bv=n(Hkv * hd))
            self.layers.append(w)

    def embed_rows(self, t):
        return self.E[np.asarray(t)]

    def layer(self, i):
        return self.layers[i]

    def lm_head(self):
        return self.lm


def _torch_rope(x, theta):
    """x [H, L, hd] -> rotate pairs (j, j + hd/2) as complex numbers by pos * theta^(-2j/hd)."""
    H, L, hd = x.shape
    half = hd // 2
    z = torch.complex(x[..., :half], x[..., half:])
    freqs = theta ** (-torch.arange(half, dtype=torch.float64) * 2 / hd)
    ang = torch.arange(L, dtype=torch.float64)[:, None] * freqs[None]
    z = z * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([z.real, z.imag], dim=-1)


def _torch_forward(w, spec, tokens, rows):
    t = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.float64)  # noqa: E731
    H, Hkv, hd = spec.n_heads, spec.n_kv_heads, spec.head_dim
    h = t(w.E)[torch.as_tensor(tokens)]
    L = h.shape[0]
    for lw in w.layers:
        a = F.rms_norm(h, (spec.d_model,), t(lw["attn_norm"]), eps=spec.rms_eps)
        q = F.linear(a, t(lw["wq"]), t(lw["bq"]) if spec.qkv_bias else None)
        k = F.linear(a, t(lw["wk"]), t(lw["bk"]) if spec.qkv_bias else None)
        v = F.linear(a, t(lw["wv"]), t(lw["bv"]) if spec.qkv_bias else None)
        q = _torch_rope(q.view(L, H, hd).transpose(0, 1), spec.rope_theta)
        k = _torch_rope(k.view(L, Hkv, hd).transpose(0, 1), spec.rope_theta)
        v = v.view(L, Hkv, hd).transpose(0, 1)
        k = k.repeat_interleave(H // Hkv, dim=0)
        v = v.repeat_interleave(H // Hkv, dim=0)
        o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=False)[0]
        h = h + F.linear(o.transpose(0, 1).reshape(L, H * hd), t(lw["wo"]))
        a = F.rms_norm(h, (spec.d_model,), t(lw["mlp_norm"]), eps=spec.rms_eps)
        h = h + F.linear(F.silu(F.linear(a, t(lw["wg"]))) * F.linear(a, t(lw["wu"])), t(lw["wd"]))
    y = F.rms_norm(h[torch.as_tensor(rows)], (spec.d_model,), t(w.final_norm), eps=spec.rms_eps)
    return (F.linear(y, t(w.lm)) * spec.logit_scale).numpy()


@pytest.mark.parametrize("kw", [{}, {"n_kv_heads": 2, "qkv_bias": True}, {"n_kv_heads": 1}])
def test_forward_matches_torch_library(kw):
    spec = _spec(**kw)
    w = _Weights(spec, 3)
    rng = np.random.default_rng(4)
    tokens = rng.integers(0, spec.vocab, (2, 13))
    rows = np.array([1, 4, 12])
    got = of.forward_logits(w, spec, tokens, rows)
    for b in range(2):
        want = _torch_forward(w, spec, tokens[b], rows)
        np.testing.assert_allclose(got[b], want, rtol=1e-10, atol=1e-10)


def test_rope_relative_position_identity():
    """<R(m) q, R(n) k> depends only on m - n."""
    rng = np.random.default_rng(0)
    hd, L = 16, 40
    q, k = rng.normal(size=hd), rng.normal(size=hd)
    cos, sin = of.rope_tables(L, hd, 1e4)
    Q = of.rope(np.tile(q, (L, 1)), cos, sin)
    K = of.rope(np.tile(k, (L, 1)), cos, sin)
    for delta in (0, 3, 17):
        vals = [Q[m] @ K[m - delta] for m in range(delta, L)]
        np.testing.assert_allclose(vals, vals[0], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(np.linalg.norm(Q, axis=1), np.linalg.norm(q), rtol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(1)
    H, L, hd = 2, 6, 4
    q = rng.normal(size=(H, L, hd))
    k = np.tile(rng.normal(size=(1, 1, hd)), (H, L, 1))       # identical keys -> uniform weights
    v = rng.normal(size=(H, L, hd))
    out = of.attention(q, k, v)
    np.testing.assert_allclose(out, np.broadcast_to(v.mean(1, keepdims=True), out.shape),
                               rtol=1e-12)
    # bidirectional: the first query sees the last key
    k2 = np.zeros((1, L, hd))
    k2[0, -1, 0] = 50.0
    q2 = np.zeros((1, L, hd))
    q2[0, :, 0] = 1.0
    out2 = of.attention(q2, k2, v[:1])
    np.testing.assert_allclose(out2[0, 0], v[0, -1], rtol=1e-6, atol=1e-6)


def test_rmsnorm_silu_closed_forms():
    x = np.array([[3.0, 4.0]])
    np.testing.assert_allclose(of.rmsnorm(x, np.ones(2), 0.0), x / np.sqrt(12.5), rtol=1e-15)
    assert of.silu(np.array([0.0]))[0] == 0.0
    assert of.silu(np.array([50.0]))[0] == pytest.approx(50.0)
