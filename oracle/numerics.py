"""Per-layer building blocks of the oracle, in float64.

The paper fixes no architecture beyond "a pretrained mask-based DLM" (LLaDA,
Dream; Sec. 3.1, Sec. 5.1).  The blocks below are the standard
LLaDA / Qwen2 decoder-layer operations, written as their plain definitions.
"""
from __future__ import annotations

import numpy as np


def round_bf16(x):
    """Round to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits (7 stored + the implicit one) and the
    float32 exponent range.  With x = m * 2**e and 0.5 <= |m| < 1, the nearest
    8-bit significand is rint(m * 2**8) (np.rint rounds half to even).
    Values below the float32 normal range keep 8 significant bits instead of
    bf16's subnormal grid; activations never get that small.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0), e - 8)


def rmsnorm(x, g, eps):
    """y = x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_angles(positions, head_dim, theta):
    """Rotation angles pos * theta^(-2i/d) for i in [0, d/2); shape [n, d/2]."""
    half = head_dim // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / head_dim)
    return np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]


def apply_rope(x, positions, theta):
    """Rotary position embedding, half-rotation pairing (i, i + d/2).

    x: [n, heads, d]; row r is at absolute position positions[r].
    x'[i]       = x[i] cos(a_i) - x[i + d/2] sin(a_i)
    x'[i + d/2] = x[i + d/2] cos(a_i) + x[i] sin(a_i)
    """
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    ang = rope_angles(positions, d, theta)[:, None, :]     # [n, 1, d/2]
    c, s = np.cos(ang), np.sin(ang)
    lo, hi = x[..., :half], x[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


def attention(q, k, v, key_valid=None):
    """Bidirectional (non-causal) scaled dot-product attention with grouped
    key/value heads.

    q: [nq, n_heads, d]; k, v: [nk, n_kv, d].  Query head h reads key/value
    head h // (n_heads / n_kv).  key_valid: optional bool [nk]; invalid keys
    get probability 0.  Returns [nq, n_heads, d].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    nq, nh, d = q.shape
    nkv = k.shape[1]
    group = nh // nkv
    out = np.empty((nq, nh, d), dtype=np.float64)
    for h in range(nh):
        g = h // group
        s = q[:, h, :] @ k[:, g, :].T / np.sqrt(d)          # [nq, nk]
        if key_valid is not None:
            s = np.where(np.asarray(key_valid)[None, :], s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out


def silu(z):
    z = np.asarray(z, dtype=np.float64)
    return z / (1.0 + np.exp(-z))


def swiglu(gate, up):
    """silu(gate) * up."""
    return silu(gate) * up
