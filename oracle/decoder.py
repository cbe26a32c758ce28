"""Plain CPU oracle of a full decoder layer for replay.  TEST INFRASTRUCTURE ONLY.

Only ``tests/`` import this module; it shares no code with
``paper_2609_04875_amd``.

The paper runs Llama-3.1-8B, Qwen2.5-7B and Mistral-7B as F (Eq. (1)) but
prints no layer; the readings follow the public architecture of those model
families (not the paper):

  D1 pre-norm decoder layer: h = RMSNorm(x) * g_attn; Q, K, V = h Wq, h Wk, h Wv;
     rotary embedding on Q and K at each token's absolute position; causal
     GQA attention over the cache (K stored rotated); x <- x + O Wo;
     h2 = RMSNorm(x) * g_mlp; x <- x + (SiLU(h2 Wg) * (h2 Wu)) Wd.  No biases.
  D2 RMSNorm(x) = x / sqrt(mean(x^2) + eps).
  D3 rotary embedding, half-split pairing: for i < d/2 the pair
     (x_i, x_{i+d/2}) turns by the angle pos * theta^(-2i/d).
  D4 SiLU(g) = g / (1 + exp(-g)).
  D5 bf16 storage points (where the GPU path stores bf16): the two norm
     outputs, Q/K/V, the rotated Q/K, the attention output, the residual
     stream after each sum, the gate and up projections, the SiLU product.
     Everything else is fp64 here.

Weights use the math layout [in][out] (x @ W).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import attention, bf16_round


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """D2 times the gain g, along the last axis, fp64."""
    x = x.astype(np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def rope(x: np.ndarray, positions: Sequence[int], theta: float) -> np.ndarray:
    """D3 on x [n, heads, d] with one absolute position per row, fp64."""
    n, _, d = x.shape
    half = d // 2
    inv = theta ** (-2.0 * np.arange(half) / d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv[None, :]     # [n, half]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half].astype(np.float64), x[..., half:].astype(np.float64)
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(g: np.ndarray) -> np.ndarray:
    """D4."""
    return g / (1.0 + np.exp(-g))


def decoder_layers(x: np.ndarray, layers: Sequence[Dict[str, np.ndarray]], n_q_heads: int, n_kv_heads: int,
                   head_dim: int, eps: float, theta: float, pos0: int = 0,
                   cache: Optional[List[Tuple[np.ndarray, np.ndarray]]] = None):
    """The tokens x [n, d_model] (fp64 holding bf16 values) at positions
    pos0 .. pos0+n-1 through every layer (D1-D5).  ``layers``: dicts with
    wq, wk, wv, wo, wg, wu, wd ([in][out]) and g_attn, g_mlp; ``cache``: per
    layer the rotated K and V of positions 0 .. pos0-1, or None when pos0 == 0.
    Returns (x_out, per-layer (K rotated, V) of the n new tokens)."""
    n = x.shape[0]
    pos = np.arange(pos0, pos0 + n)
    scale = head_dim ** -0.5
    new_kv = []
    for li, w in enumerate(layers):
        h = bf16_round(rms_norm(x, w["g_attn"], eps))
        q = bf16_round(h @ w["wq"]).reshape(n, n_q_heads, head_dim)
        k = bf16_round(h @ w["wk"]).reshape(n, n_kv_heads, head_dim)
        v = bf16_round(h @ w["wv"]).reshape(n, n_kv_heads, head_dim)
        q = bf16_round(rope(q, pos, theta))
        k = bf16_round(rope(k, pos, theta))
        if pos0 > 0:
            kc, vc = cache[li]
            kk, vv = np.concatenate([kc[:pos0], k]), np.concatenate([vc[:pos0], v])
        else:
            kk, vv = k, v
        o = bf16_round(attention(q, kk, vv, pos0, scale)).reshape(n, n_q_heads * head_dim)
        x = bf16_round(x + o @ w["wo"])
        h2 = bf16_round(rms_norm(x, w["g_mlp"], eps))
        g = bf16_round(h2 @ w["wg"])
        u = bf16_round(h2 @ w["wu"])
        a = bf16_round(silu(g) * u)
        x = bf16_round(x + a @ w["wd"])
        new_kv.append((k, v))
    return x, new_kv
