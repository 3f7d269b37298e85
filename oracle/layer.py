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
* A Llama-style decoder layer over one serving iteration: the steps above and
  the attention oracle in float64, with each tensor that the boundary stores in
  bf16 rounded to bf16 (round to nearest, ties to even, straight from float64)
  where it is stored.
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


def bf16_round(x) -> np.ndarray:
    """float64 values rounded to the nearest bf16 (8 significant bits), ties to
    even, with no intermediate float32 step."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)  # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def bf16_bits(x) -> np.ndarray:
    """bf16 bit patterns (uint16) of values that are already bf16-exact."""
    y = np.asarray(x, dtype=np.float64).astype(np.float32)
    return (y.view(np.uint32) >> 16).astype(np.uint16)


def from_bits(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def decoder_layer(x, wts, hq, hkv, d, q_len, ctx_len, block_table, k_cache, v_cache, eps,
                  base=500000.0, scale=None):
    """One decoder layer over the new tokens of a batch B = {(c_i, u_i)}.

    x [T, hidden] and the weights (dict: attn_norm, w_q, w_k, w_v, w_o, mlp_norm,
    w_gate, w_up, w_down, as bf16 bit arrays) are bf16; k_cache / v_cache are the
    pools before the iteration (bf16 bits).  Returns (out [T, hidden] float64,
    bf16-exact; the pools after the append)."""
    from oracle import oracle as attn_oracle  # the attention and kv_append oracle
    f = {k: from_bits(v) for k, v in wts.items()}
    xf = from_bits(x)
    t = xf.shape[0]
    pos = positions(q_len, ctx_len)
    xn = bf16_round(rms_norm(xf, f["attn_norm"], eps))
    q = bf16_round(linear(xn, f["w_q"])).reshape(t, hq, d)
    k = bf16_round(linear(xn, f["w_k"])).reshape(t, hkv, d)
    v = bf16_round(linear(xn, f["w_v"])).reshape(t, hkv, d)
    q = bf16_round(rope(q, pos, base))
    k = bf16_round(rope(k, pos, base))
    kc, vc = attn_oracle.kv_append(hkv, d, 16, q_len, ctx_len, block_table, bf16_bits(k),
                                   bf16_bits(v), k_cache, v_cache)
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    a, _ = attn_oracle.attention(hq, hkv, d, 16, scale, q_len, ctx_len, block_table, bf16_bits(q),
                                 kc, vc)
    a = bf16_round(a.reshape(t, hq * d))
    h = bf16_round(xf + linear(a, f["w_o"]))
    hn = bf16_round(rms_norm(h, f["mlp_norm"], eps))
    act = bf16_round(silu_mul(linear(hn, f["w_gate"]), linear(hn, f["w_up"])))
    out = bf16_round(h + linear(act, f["w_down"]))
    return out, kc, vc
