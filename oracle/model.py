"""The masked-diffusion LM forward, as the oracle computes it (float64).

Two entry points:

* ``forward``       - the plain full forward F of a bidirectional decoder over
  a token prefix (each diffusion step of standard DLM inference runs it over
  the whole sequence, Sec. 3.1; the refresh step runs it over the phase's
  retained tokens, Sec. 4.3, refresh equation).  It also returns every
  layer's K and V, which is what the refresh writes into the cache.
* ``forward_rows``  - the normal-step forward of Sec. 4.3: only the online
  rows (active tokens and tokens decoded inside the phase) are computed; at
  every layer their fresh K/V overwrite their cache rows, and they attend to
  all cache rows of the retained prefix, whose other rows (earlier-decoded
  context and buffer tokens) still hold the K/V of the last refresh.

Layer layout (the paper gives none; this is the LLaDA / Qwen2 layer):
pre-RMSNorm, Q/K/V projections (+bias for Qwen2-style models), RoPE on Q and
K at absolute positions, non-causal attention, output projection, residual;
pre-RMSNorm, SwiGLU FFN, residual; final RMSNorm and an untied LM head.

bf16 models: the weights are bf16 values (exact in float64).  The residual
stream is not rounded.  These intermediate tensors are rounded to bf16,
which is where the GPU datapath stores bf16: both RMSNorm outputs, Q and K
after RoPE, V, the attention output and the SwiGLU product.  Everything else
(accumulations, softmax, logits) stays float64 here.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

import synth
from .numerics import apply_rope, attention, rmsnorm, round_bf16, swiglu


def _identity(x):
    return x


class KVCache:
    """Per-layer K and V rows at absolute positions: K[l] is [S, n_kv, d].
    Rows never written hold NaN, so reading one poisons the result."""

    def __init__(self, n_layers: int, seq_len: int, n_kv: int, head_dim: int):
        self.K = [np.full((seq_len, n_kv, head_dim), np.nan) for _ in range(n_layers)]
        self.V = [np.full((seq_len, n_kv, head_dim), np.nan) for _ in range(n_layers)]

    def copy(self) -> "KVCache":
        c = KVCache.__new__(KVCache)
        c.K = [k.copy() for k in self.K]
        c.V = [v.copy() for v in self.V]
        return c


# the projection matrices that the FP8-weight variant stores as e4m3
FP8_MATRICES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "lm_head")


class OracleModel:
    """float64 reference model over ``synth.Weights``.

    ``cache_budget_bytes`` bounds how many float64 weight tensors stay in
    memory; beyond it tensors are re-read from the seeded generator on use.
    ``weight_format="fp8"`` (bf16 models only) is the FP8-weight variant: the
    projection matrices are replaced by their per-row e4m3 quantization
    (oracle.quant); embeddings, norm gains and biases stay bf16.
    """

    def __init__(self, weights: synth.Weights, cache_budget_bytes: float = 8e9,
                 weight_format: str = "bf16"):
        if weight_format not in ("bf16", "fp8"):
            raise ValueError("weight_format is 'bf16' or 'fp8'")
        if weight_format == "fp8" and weights.shape.dtype != synth.DTYPE_BF16:
            raise ValueError("FP8 weights are a variant of bf16 models")
        self.weight_format = weight_format
        self.shape = weights.shape
        self.weights = weights
        self.bf16 = self.shape.dtype == synth.DTYPE_BF16
        self.rnd = round_bf16 if self.bf16 else _identity
        self._budget = cache_budget_bytes
        self._used = 0
        self._cache: Dict[str, np.ndarray] = {}
        self._emb_raw: Optional[np.ndarray] = None

    # -- weights ---------------------------------------------------------
    def w(self, name: str) -> np.ndarray:
        t = self._cache.get(name)
        if t is not None:
            return t
        if self.weight_format == "fp8" and name.split(".")[-1] in FP8_MATRICES:
            from .quant import dequantize_rows, quantize_rows
            t = dequantize_rows(*quantize_rows(self.weights.f32(name)))
        else:
            t = self.weights.f32(name).astype(np.float64)
        if self._used + t.nbytes <= self._budget:
            self._cache[name] = t
            self._used += t.nbytes
        return t

    def emb_rows(self, ids) -> np.ndarray:
        if self._emb_raw is None:
            self._emb_raw = self.weights.f32("emb")
        return self._emb_raw[np.asarray(ids, dtype=np.int64)].astype(np.float64)

    # -- one decoder layer ----------------------------------------------
    def _qkv(self, l: int, h: np.ndarray, pos: np.ndarray):
        m = self.shape
        p = f"layers.{l}."
        n = h.shape[0]
        a = self.rnd(rmsnorm(h, self.w(p + "attn_norm"), m.rms_eps))
        q = a @ self.w(p + "wq").T
        k = a @ self.w(p + "wk").T
        v = a @ self.w(p + "wv").T
        if m.qkv_bias:
            q = q + self.w(p + "bq")
            k = k + self.w(p + "bk")
            v = v + self.w(p + "bv")
        q = self.rnd(apply_rope(q.reshape(n, m.n_heads, m.head_dim), pos, m.rope_theta))
        k = self.rnd(apply_rope(k.reshape(n, m.n_kv_heads, m.head_dim), pos, m.rope_theta))
        v = self.rnd(v.reshape(n, m.n_kv_heads, m.head_dim))
        return q, k, v

    def _after_attention(self, l: int, h: np.ndarray, o: np.ndarray) -> np.ndarray:
        m = self.shape
        p = f"layers.{l}."
        n = h.shape[0]
        o = self.rnd(o.reshape(n, m.q_dim))
        h = h + o @ self.w(p + "wo").T
        a = self.rnd(rmsnorm(h, self.w(p + "ffn_norm"), m.rms_eps))
        s = self.rnd(swiglu(a @ self.w(p + "wg").T, a @ self.w(p + "wu").T))
        return h + s @ self.w(p + "wd").T

    # -- forwards ----------------------------------------------------------
    def forward(self, ids: Sequence[int], positions: Optional[Sequence[int]] = None,
                n_layers: Optional[int] = None):
        """Full bidirectional forward F over ``ids`` (every token attends to
        every token).  Returns (h_final [n, H] before the final norm,
        K list, V list) with K[l], V[l] of shape [n, n_kv, d]."""
        n = len(ids)
        pos = np.arange(n) if positions is None else np.asarray(positions)
        h = self.emb_rows(ids)
        Ks: List[np.ndarray] = []
        Vs: List[np.ndarray] = []
        for l in range(self.shape.n_layers if n_layers is None else n_layers):
            q, k, v = self._qkv(l, h, pos)
            Ks.append(k)
            Vs.append(v)
            h = self._after_attention(l, h, attention(q, k, v))
        return h, Ks, Vs

    def forward_rows(self, ids_rows: Sequence[int], pos_rows: Sequence[int],
                     cache: KVCache, ctx_len: int, n_layers: Optional[int] = None):
        """Normal-step forward of the rows at absolute positions ``pos_rows``
        (all < ctx_len).  At each layer their fresh K/V overwrite the cache at
        their positions, then they attend to cache rows [0, ctx_len).
        Returns h_final [len(rows), H] before the final norm."""
        pos = np.asarray(pos_rows, dtype=np.int64)
        assert pos.size == 0 or int(pos.max()) < ctx_len
        h = self.emb_rows(ids_rows)
        for l in range(self.shape.n_layers if n_layers is None else n_layers):
            q, k, v = self._qkv(l, h, pos)
            cache.K[l][pos] = k
            cache.V[l][pos] = v
            o = attention(q, cache.K[l][:ctx_len], cache.V[l][:ctx_len])
            h = self._after_attention(l, h, o)
        return h

    def logits(self, h_rows: np.ndarray) -> np.ndarray:
        """Final RMSNorm and LM head: [n, H] -> [n, vocab]."""
        a = self.rnd(rmsnorm(h_rows, self.w("final_norm"), self.shape.rms_eps))
        return a @ self.w("lm_head").T

    def new_cache(self, seq_len: int) -> KVCache:
        m = self.shape
        return KVCache(m.n_layers, seq_len, m.n_kv_heads, m.head_dim)
