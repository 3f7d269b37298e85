"""CPU oracle of the layer steps around attention (include/ssa_layer.h).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, never by the library.  Plain
numpy in float64; it imports nothing from the library package.

* Positions of the new tokens: token j of request i sits at u_i + j (Sec. 3.2's
  batch B = {(c_i, u_i)}: c_i new tokens after u_i cached ones).
* Rotary position embedding, "rotate half" pairing, as in Llama: for dims
  i < D/2 of a head, with angle a = p * base^(-2i/D),
      out[i] = x[i] cos a - x[i + D/2] sin a,  out[i + D/2] = x[i + D/2] cos a + x[i] sin a.
  Angles and products in float64.
* A linear layer: x W^T for W stored [out features, in features].
* RMSNorm: x / sqrt(mean(x^2) + eps) * weight.
* SwiGLU: silu(gate) * up with silu(z) = z / (1 + exp(-z)).
"""
from __future__ import annotations

import numpy as np


def positions(q_len, ctx_len) -> np.ndarray:
    """Position of every new token, in request order."""
    return np.concatenate([np.arange(u, u + c, dtype=np.int64)
                           for c, u in zip(q_len, ctx_len)] or [np.zeros(0, np.int64)])


def rope(x, pos, base: float = 500000.0) -> np.ndarray:
    """x [T, H, D] (float64), pos [T]: the rotated heads."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv = base ** (-2.0 * np.arange(half, dtype=np.float64) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]  # [T, D/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def linear(x, w) -> np.ndarray:
    """x [M, K], w [N, K]: x w^T in float64."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T


def rms_norm(x, weight, eps: float = 1e-5) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(weight, np.float64)


def silu_mul(gate, up) -> np.ndarray:
    g = np.asarray(gate, dtype=np.float64)
    return g / (1.0 + np.exp(-g)) * np.asarray(up, dtype=np.float64)
