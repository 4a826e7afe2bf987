"""Oracle dense forward pass (test infrastructure only).

The method keeps the backbone frozen and runs one dense Transformer pass per
executed step (Section 3, Method, first paragraph).  The paper does not spell
out the backbone; the pass here is the standard bidirectional masked-diffusion
LM that LLaDA and Dream use:

    h = E[x]
    per layer:  a = rmsnorm(h);  q, k, v = a Wq^T (+bq), a Wk^T (+bk), a Wv^T (+bv)
                q, k = rope(q), rope(k)                 (rotate-half, positions 0..L-1)
                o = softmax(q k^T / sqrt(hd)) v         (no mask: every position sees all)
                h = h + o Wo^T
                a = rmsnorm(h);  h = h + (silu(a Wg^T) * (a Wu^T)) Wd^T
    logits[rows] = rmsnorm(h)[rows] Wlm^T * logit_scale

Weights arrive as an object with ``embed_rows(tokens)``, ``layer(i)`` (dict of
``wq wk wv wo wg wu wd`` [out, in] and optional ``bq bk bv``, ``attn_norm``,
``mlp_norm``), ``lm_head()`` [V, d] and ``final_norm``.  All arithmetic is in
``dtype`` (fp64 by default) with no intermediate rounding.
"""
import numpy as np


def rmsnorm(x, w, eps):
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def rope_tables(L, hd, theta, dtype=np.float64):
    """cos and sin of pos * theta^(-2j/hd), pos = 0..L-1, j = 0..hd/2-1 (fp64)."""
    j = np.arange(hd // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * j / hd)
    ang = np.arange(L, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang).astype(dtype), np.sin(ang).astype(dtype)


def rope(x, cos, sin):
    """Rotate-half RoPE on the last axis of x [..., L, hd]: dims j and j + hd/2 form a pair."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def softmax(s, axis=-1):
    s = s - np.max(s, axis=axis, keepdims=True)
    e = np.exp(s)
    return e / np.sum(e, axis=axis, keepdims=True)


def attention(q, k, v):
    """Bidirectional attention.  q [H, L, hd], k/v [Hkv, L, hd]; query head j reads kv head
    j // (H / Hkv).  No mask."""
    H, L, hd = q.shape
    Hkv = k.shape[0]
    group = H // Hkv
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for j in range(H):
        kv = j // group
        p = softmax((q[j] @ k[kv].T) * scale)
        out[j] = p @ v[kv]
    return out


def silu(x):
    return x / (1.0 + np.exp(-x))


def layer_forward(h, w, spec, cos, sin, dtype):
    """One pre-norm residual block on h [L, d] (one sequence)."""
    L, d = h.shape
    H, Hkv, hd = spec.n_heads, spec.n_kv_heads, spec.head_dim
    W = lambda n: np.asarray(w[n], dtype=dtype)  # noqa: E731
    a = rmsnorm(h, W("attn_norm"), spec.rms_eps)
    q, k, v = a @ W("wq").T, a @ W("wk").T, a @ W("wv").T
    if spec.qkv_bias:
        q, k, v = q + W("bq"), k + W("bk"), v + W("bv")
    q = q.reshape(L, H, hd).transpose(1, 0, 2)
    k = k.reshape(L, Hkv, hd).transpose(1, 0, 2)
    v = v.reshape(L, Hkv, hd).transpose(1, 0, 2)
    q, k = rope(q, cos, sin), rope(k, cos, sin)
    o = attention(q, k, v).transpose(1, 0, 2).reshape(L, H * hd)
    h = h + o @ W("wo").T
    a = rmsnorm(h, W("mlp_norm"), spec.rms_eps)
    u = silu(a @ W("wg").T) * (a @ W("wu").T)
    return h + u @ W("wd").T


def hidden_states(weights, spec, tokens, dtype=np.float64):
    """Final residual stream h [B, L, d] for tokens [B, L]."""
    tokens = np.asarray(tokens)
    B, L = tokens.shape
    cos, sin = rope_tables(L, spec.head_dim, spec.rope_theta, dtype)
    hs = np.stack([np.asarray(weights.embed_rows(tokens[b]), dtype=dtype) for b in range(B)])
    for i in range(spec.n_layers):
        w = weights.layer(i)
        for b in range(B):
            hs[b] = layer_forward(hs[b], w, spec, cos, sin, dtype)
    return hs


def logits_from_hidden(weights, spec, h_rows, dtype=np.float64):
    """LM head on selected rows: rmsnorm(h) Wlm^T * logit_scale."""
    y = rmsnorm(h_rows, np.asarray(weights.final_norm, dtype=dtype), spec.rms_eps)
    return (y @ np.asarray(weights.lm_head(), dtype=dtype).T) * spec.logit_scale


def forward_logits(weights, spec, tokens, rows, dtype=np.float64):
    """Logits [B, len(rows_b), V] of canvas positions rows[b] (a list/array per batch row,
    or one array used for every row)."""
    tokens = np.asarray(tokens)
    B = tokens.shape[0]
    hs = hidden_states(weights, spec, tokens, dtype)
    out = []
    for b in range(B):
        r = rows[b] if isinstance(rows, (list, tuple)) else rows
        out.append(logits_from_hidden(weights, spec, hs[b][np.asarray(r)], dtype))
    return np.stack(out)
