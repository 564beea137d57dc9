"""float64 building blocks of a Llama-style decoder (oracle side).

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (8 significant bits,
    ties to even), returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                  # x = m * 2**e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


class Numerics:
    """Where values are stored at reduced precision.

    "f32": the fp32 configuration; the oracle keeps everything in float64
    (the GPU's fp32 differs only by rounding, inside the 1e-4 tolerance).
    "bf16": the bf16 configurations store weights, the inputs of every
    projection (A operand), Q/K/V after RoPE and the attention output in
    bfloat16 and accumulate in fp32; ``act`` applies that rounding here.
    """

    def __init__(self, dtype: str):
        if dtype not in ("f32", "bf16"):
            raise ValueError(dtype)
        self.dtype = dtype

    def act(self, x):
        return round_bf16(x) if self.dtype == "bf16" else np.asarray(
            x, dtype=np.float64)


def rmsnorm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x):
    return x / (1.0 + np.exp(-x))


def rope(x, pos, theta):
    """Rotary embedding, rotate-half pairing (i, i + hd/2).

    x: [..., n_heads, hd]; pos: integer positions broadcastable to x[..., 0, 0].
    """
    hd = x.shape[-1]
    half = hd // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv      # [..., half]
    c = np.cos(ang)[..., None, :]
    s = np.sin(ang)[..., None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s):
    s = np.asarray(s, dtype=np.float64)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def logsumexp(z):
    z = np.asarray(z, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    return (m + np.log(np.exp(z - m).sum(axis=-1, keepdims=True)))[..., 0]


def attend(q, keys, vals):
    """Softmax attention of one query row over an explicit key set.

    q: [H, hd]; keys, vals: [n, Hkv, hd] (n >= 1).  Query head h reads KV head
    h // (H / Hkv) (grouped-query attention); scores are scaled by 1/sqrt(hd).
    Returns [H * hd].
    """
    H, hd = q.shape
    group = H // keys.shape[1]
    out = np.empty((H, hd))
    for h in range(H):
        kh = h // group
        p = softmax(keys[:, kh, :] @ q[h] / np.sqrt(hd))
        out[h] = p @ vals[:, kh, :]
    return out.reshape(-1)
