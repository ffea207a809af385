"""The controlled analysis behind Observation 2 (Sec. 3.2): how much the
active tokens' predictions depend on the undecoded context, and how well the
non-active masked tokens' K/V can be reused.  A functional experiment on
the oracle model (random weights here, so its numbers say nothing about
trained models); test infrastructure like the rest of the oracle.

At an observation step t0 the active set A is the first n_active (16 in the
paper) undecoded positions.  The reference is the full-sequence, no-cache
prediction of A.  For each W, the visible context is every decoded position
plus the first W undecoded positions (the undecoded context truncated to a
prefix of length W, A included), and two configurations are scored by the
KL divergence of A's predictions from the reference, averaged over A:

* truncation only: a plain forward over the visible context;
* truncation + cache: the same context, but the non-active masked tokens
  of it keep the K/V they had at step t0 - 1 (from the same truncated
  forward over the state of step t0 - 1); decoded and active tokens are
  recomputed.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np

from .model import OracleModel
from .numerics import attention


def _softmax_predictions(model: OracleModel, h: np.ndarray) -> np.ndarray:
    """Predictive distribution of rows h ([MASK] excluded), float64."""
    logits = model.logits(h)
    logits[:, model.shape.mask_id] = -np.inf
    logits = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(logits)
    return p / p.sum(axis=1, keepdims=True)


def _forward_subset(model: OracleModel, x: np.ndarray, rows: Sequence[int],
                    cached: Dict[int, List[np.ndarray]] = None,
                    keep: Sequence[int] = ()):
    """Forward over the visible positions `rows` (absolute positions, RoPE
    at those positions, every row attends to every visible row).  Rows listed
    in `keep` take their K/V at every layer from `cached[l]` (indexed like
    `rows`) instead of computing them.  Returns (h [len(rows), H], K, V per
    layer)."""
    rows = list(rows)
    pos = np.asarray(rows)
    keep_idx = [rows.index(p) for p in keep]
    h = model.emb_rows(x[pos])
    Ks, Vs = [], []
    for l in range(model.shape.n_layers):
        q, k, v = model._qkv(l, h, pos)
        if keep_idx:
            k[keep_idx] = cached["K"][l][keep_idx]
            v[keep_idx] = cached["V"][l][keep_idx]
        Ks.append(k)
        Vs.append(v)
        h = model._after_attention(l, h, attention(q, k, v))
    return h, Ks, Vs


def kl_rows(p: np.ndarray, q: np.ndarray) -> np.ndarray:
    """KL(p || q) per row, in nats."""
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(p > 0, p * (np.log(p) - np.log(q)), 0.0)
    return t.sum(axis=1)


def observation2(model: OracleModel, x_prev: np.ndarray, x: np.ndarray,
                 decoded: np.ndarray, widths: Sequence[int], n_active: int = 16) -> Dict:
    """KL of the active predictions from the full no-cache reference, per W.

    x_prev / x: the token sequences at steps t0 - 1 and t0 (x_prev may hold
    [MASK] at positions decoded at step t0 - 1); decoded: the decoded flags
    at t0.  Returns {"active": A, "W": [...], "truncation": [...],
    "truncation_cache": [...]} with the mean KL over A for each W."""
    S = len(x)
    und = [int(i) for i in np.flatnonzero(~decoded)]
    A = und[:n_active]
    dec = [int(i) for i in np.flatnonzero(decoded)]
    h_ref, _, _ = _forward_subset(model, x, list(range(S)))
    ref = _softmax_predictions(model, h_ref[A])
    out = {"active": A, "W": [], "truncation": [], "truncation_cache": []}
    for W in widths:
        if W < len(A):
            continue
        rows = sorted(dec + und[:W])
        idx = [rows.index(p) for p in A]
        h_t, _, _ = _forward_subset(model, x, rows)
        kl_t = kl_rows(ref, _softmax_predictions(model, h_t[idx])).mean()
        # K/V of the step before, over the same visible positions
        _, Kp, Vp = _forward_subset(model, x_prev, rows)
        buffer = [p for p in und[:W] if p not in A]
        h_c, _, _ = _forward_subset(model, x, rows, {"K": Kp, "V": Vp}, keep=buffer)
        kl_c = kl_rows(ref, _softmax_predictions(model, h_c[idx])).mean()
        out["W"].append(W)
        out["truncation"].append(float(kl_t))
        out["truncation_cache"].append(float(kl_c))
    return out
