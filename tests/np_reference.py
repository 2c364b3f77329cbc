"""An independent float64 numpy composition of the decoder, used only to pin
the oracle's forward. It is written as whole-sequence matrix products with a
causal mask and RoPE as a complex rotation, so it shares no structure with the
oracle's row-at-a-time fp32 loops."""
from __future__ import annotations

import numpy as np

import synth


def rope_phases(shape: synth.ModelShape, n_pos: int) -> np.ndarray:
    """Complex phases [n_pos, dh/2] for positions 0..n_pos-1 (position 0 unturned,
    positions beyond T clamped to T). Pairs below dh/4 turn with the grid row,
    the others with the grid column."""
    dh, G = shape.head_dim, shape.grid
    quarter = dh // 4
    theta = shape.rope_base ** (-4.0 * np.arange(quarter) / dh)
    out = np.ones((n_pos, dh // 2), dtype=np.complex128)
    for s in range(1, n_pos):
        g = min(s, shape.T) - 1
        row, col = divmod(g, G)
        ang = np.concatenate([row * theta, col * theta])
        out[s] = np.exp(1j * ang)
    return out


def apply_rope(x: np.ndarray, phases: np.ndarray) -> np.ndarray:
    """x [n, heads, dh] -> rotated copy."""
    z = x[..., 0::2] + 1j * x[..., 1::2]
    z = z * phases[:, None, :]
    out = np.empty_like(x)
    out[..., 0::2] = z.real
    out[..., 1::2] = z.imag
    return out


def rms(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def forward(shape: synth.ModelShape, blob: np.ndarray, cls: int, tokens) -> np.ndarray:
    """Logits [(n+1), V] for [class, x_1..x_n], float64 throughout."""
    W = {k: v.astype(np.float64) for k, v in synth.split_blob(shape, blob).items()}
    tokens = np.asarray(tokens, dtype=np.int64)
    n = tokens.size + 1
    H, dh, d = shape.n_heads, shape.head_dim, shape.d_model
    x = np.concatenate([W["cls_emb"][cls][None, :], W["tok_emb"][tokens]], axis=0)
    ph = rope_phases(shape, n)
    mask = np.tril(np.ones((n, n), dtype=bool))
    for layer in range(shape.n_layers):
        p = f"l{layer}."
        a = rms(x, W[p + "g_attn"], shape.rms_eps)
        qkv = a @ W[p + "wqkv"].T
        q = apply_rope(qkv[:, :d].reshape(n, H, dh), ph)
        k = apply_rope(qkv[:, d:2 * d].reshape(n, H, dh), ph)
        v = qkv[:, 2 * d:].reshape(n, H, dh)
        s = np.einsum("ihe,jhe->hij", q, k) / np.sqrt(dh)
        s = np.where(mask[None], s, -np.inf)
        s = s - s.max(axis=-1, keepdims=True)
        e = np.exp(s)
        att = e / e.sum(axis=-1, keepdims=True)
        o = np.einsum("hij,jhe->ihe", att, v).reshape(n, d)
        x = x + o @ W[p + "wo"].T
        m = rms(x, W[p + "g_ffn"], shape.rms_eps)
        g = m @ W[p + "w1"].T
        u = m @ W[p + "w3"].T
        x = x + (g / (1.0 + np.exp(-g)) * u) @ W[p + "w2"].T
    logits = rms(x, W["g_out"], shape.rms_eps) @ W["w_lm"].T
    if shape.has_lm_bias:
        logits = logits + W["b_lm"]
    return logits


def softmax_topk(l: np.ndarray, tau: float, k: int) -> np.ndarray:
    """float64 softmax of l / tau restricted to the entries >= the k-th largest."""
    y = np.asarray(l, dtype=np.float64) / tau
    keep = np.ones_like(y, dtype=bool)
    if 0 < k < y.size:
        thr = np.sort(y)[::-1][k - 1]
        keep = y >= thr
    e = np.where(keep, np.exp(y - y[keep].max()), 0.0)
    return e / e.sum()
