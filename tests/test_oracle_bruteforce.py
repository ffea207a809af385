"""Pin of the oracle forward: an independent pure-Python (float64, explicit
loops, math module) implementation of the same decoder layer, on micro
models, must agree with the NumPy oracle to round-off.

The loop version is written from the layer definitions, not from the
oracle's code: per-element dot products, per-pair rotations, per-key
softmax.  A transposed weight, a wrong GQA head map, a RoPE pairing or sign
slip, a missing residual or bias in either implementation fails here.
"""
import math

import numpy as np
import pytest

import synth
from oracle.model import OracleModel


def micro_shape(dtype, bias, n_kv=2):
    return synth.ModelShape(n_layers=2, hidden=32, n_heads=4, n_kv_heads=n_kv, head_dim=8,
                            ffn=48, vocab=50, dtype=dtype, qkv_bias=bias, rms_eps=1e-5,
                            rope_theta=100.0)


def rne_bf16(x):
    """Nearest value with 8 significant bits, ties to even (Python's round)."""
    if x == 0.0:
        return 0.0
    m, e = math.frexp(x)
    return math.ldexp(round(m * 256.0), e - 8)


class LoopModel:
    def __init__(self, W: synth.Weights):
        self.s = W.shape
        self.t = {name: W.f32(name).astype(np.float64).tolist() for name, _, _ in W.specs}
        self.r = rne_bf16 if self.s.dtype == synth.DTYPE_BF16 else (lambda v: v)

    def linear(self, x, name, bias=None):
        Wt = self.t[name]
        out = []
        for o in range(len(Wt)):
            acc = 0.0
            for i in range(len(x)):
                acc += x[i] * Wt[o][i]
            if bias is not None:
                acc += self.t[bias][o]
            out.append(acc)
        return out

    def norm(self, x, g):
        ms = sum(v * v for v in x) / len(x)
        inv = 1.0 / math.sqrt(ms + self.s.rms_eps)
        return [self.r(x[i] * inv * self.t[g][i]) for i in range(len(x))]

    def rope(self, vec, pos):
        d = len(vec)
        half = d // 2
        out = [0.0] * d
        for i in range(half):
            a = pos * self.s.rope_theta ** (-2.0 * i / d)
            out[i] = vec[i] * math.cos(a) - vec[i + half] * math.sin(a)
            out[i + half] = vec[i + half] * math.cos(a) + vec[i] * math.sin(a)
        return out

    def qkv(self, l, h, pos):
        s = self.s
        p = f"layers.{l}."
        a = self.norm(h, p + "attn_norm")
        bq, bk, bv = ((p + "bq", p + "bk", p + "bv") if s.qkv_bias else (None, None, None))
        q = self.linear(a, p + "wq", bq)
        k = self.linear(a, p + "wk", bk)
        v = self.linear(a, p + "wv", bv)
        d = s.head_dim
        qh = [[self.r(z) for z in self.rope(q[h * d:(h + 1) * d], pos)] for h in range(s.n_heads)]
        kh = [[self.r(z) for z in self.rope(k[h * d:(h + 1) * d], pos)] for h in range(s.n_kv_heads)]
        vh = [[self.r(z) for z in v[h * d:(h + 1) * d]] for h in range(s.n_kv_heads)]
        return qh, kh, vh

    def attend(self, qh, Ks, Vs):
        """qh: [heads][d] of one row; Ks/Vs: per key [kv_heads][d]."""
        s = self.s
        d = s.head_dim
        out = []
        for h in range(s.n_heads):
            g = h * s.n_kv_heads // s.n_heads
            scores = [sum(qh[h][i] * K[g][i] for i in range(d)) / math.sqrt(d) for K in Ks]
            mx = max(scores)
            e = [math.exp(z - mx) for z in scores]
            tot = sum(e)
            for i in range(d):
                out.append(self.r(sum(e[j] * Vs[j][g][i] for j in range(len(Ks))) / tot))
        return out

    def rest(self, l, h, o):
        p = f"layers.{l}."
        ao = self.linear(o, p + "wo")
        h = [h[i] + ao[i] for i in range(len(h))]
        a = self.norm(h, p + "ffn_norm")
        g = self.linear(a, p + "wg")
        u = self.linear(a, p + "wu")
        sw = [self.r(g[i] / (1.0 + math.exp(-g[i])) * u[i]) for i in range(len(g))]
        dn = self.linear(sw, p + "wd")
        return [h[i] + dn[i] for i in range(len(h))]

    def forward(self, ids):
        n = len(ids)
        hs = [list(self.t["emb"][t]) for t in ids]
        kv = []
        for l in range(self.s.n_layers):
            per = [self.qkv(l, hs[r], r) for r in range(n)]
            Ks = [x[1] for x in per]
            Vs = [x[2] for x in per]
            kv.append((Ks, Vs))
            hs = [self.rest(l, hs[r], self.attend(per[r][0], Ks, Vs)) for r in range(n)]
        return hs, kv

    def forward_rows(self, ids_rows, pos_rows, kv, ctx):
        """Rows attend to cache rows [0, ctx) after overwriting their own."""
        hs = [list(self.t["emb"][t]) for t in ids_rows]
        for l in range(self.s.n_layers):
            Ks = [list(r) for r in kv[l][0]]
            Vs = [list(r) for r in kv[l][1]]
            per = [self.qkv(l, hs[i], pos_rows[i]) for i in range(len(hs))]
            for i, p in enumerate(pos_rows):
                Ks[p] = per[i][1]
                Vs[p] = per[i][2]
            kv[l] = (Ks, Vs)
            hs = [self.rest(l, hs[i], self.attend(per[i][0], Ks[:ctx], Vs[:ctx]))
                  for i in range(len(hs))]
        return hs

    def logits(self, h):
        a = self.norm(h, "final_norm")
        return self.linear(a, "lm_head")


CASES = [(synth.DTYPE_F32, False, 2), (synth.DTYPE_F32, True, 4), (synth.DTYPE_BF16, True, 2),
         (synth.DTYPE_BF16, False, 1)]


@pytest.mark.parametrize("dtype,bias,n_kv", CASES)
def test_full_forward_matches_loops(dtype, bias, n_kv):
    shape = micro_shape(dtype, bias, n_kv)
    W = synth.Weights(shape, seed=7, std=0.2)
    rng = np.random.default_rng(3)
    ids = rng.integers(0, shape.vocab, size=9).tolist()
    om = OracleModel(W)
    h, K, V = om.forward(ids)
    lg = om.logits(h)
    lm = LoopModel(W)
    hb, kvb = lm.forward(ids)
    lgb = np.array([lm.logits(r) for r in hb])
    np.testing.assert_allclose(h, np.array(hb), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lg, lgb, rtol=1e-12, atol=1e-12)
    for l in range(shape.n_layers):
        np.testing.assert_allclose(K[l], np.array(kvb[l][0]), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(V[l], np.array(kvb[l][1]), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("dtype,bias,n_kv", CASES[:3])
def test_row_forward_matches_loops(dtype, bias, n_kv):
    """Normal-step forward: rows {1, 4, 5} of a 8-token prefix recomputed over a
    cache that holds stale K/V from different tokens."""
    shape = micro_shape(dtype, bias, n_kv)
    W = synth.Weights(shape, seed=11, std=0.2)
    rng = np.random.default_rng(5)
    ids_old = rng.integers(0, shape.vocab, size=8).tolist()
    ids_new = list(ids_old)
    rows = [1, 4, 5]
    for r in rows:
        ids_new[r] = int(rng.integers(0, shape.vocab))
    ctx = 7
    om = OracleModel(W)
    _, K, V = om.forward(ids_old)
    cache = om.new_cache(8)
    for l in range(shape.n_layers):
        cache.K[l][:] = K[l]
        cache.V[l][:] = V[l]
    h = om.forward_rows([ids_new[r] for r in rows], rows, cache, ctx)
    lm = LoopModel(W)
    _, kvb = lm.forward(ids_old)
    hb = lm.forward_rows([ids_new[r] for r in rows], rows, kvb, ctx)
    np.testing.assert_allclose(h, np.array(hb), rtol=1e-12, atol=1e-12)
    for l in range(shape.n_layers):
        np.testing.assert_allclose(cache.K[l], np.array(kvb[l][0]), rtol=1e-12, atol=1e-12)
