"""The Observation 2 probe (oracle.probe) on a small random model: a
functional check of the experiment's structure (random weights carry no
meaning for its numbers), pinned by the cases that have a known answer."""
import numpy as np

import synth
from oracle.model import OracleModel
from oracle.probe import _forward_subset, kl_rows, observation2
from oracle.schedule import FullDecoder


def _state(model, prompt, G, t0, k=2):
    """Full decoding to step t0: tokens at t0 - 1 and t0, decoded flags at t0."""
    dec = FullDecoder(model, prompt, G, k)
    for _ in range(t0 - 1):
        dec.step()
    x_prev = dec.x.copy()
    dec.step()
    return x_prev, dec.x.copy(), dec.decoded.copy()


def test_observation2_probe_structure():
    shape = synth.ModelShape(n_layers=2, hidden=64, n_heads=4, n_kv_heads=2, head_dim=16,
                             ffn=96, vocab=80, dtype=synth.DTYPE_F32, rope_theta=100.0)
    m = OracleModel(synth.Weights(shape, seed=4, std=0.3))
    prompt = [3, 14, 15, 9, 26, 5]
    G = 40
    x_prev, x, decoded = _state(m, prompt, G, t0=4)
    n_und = int((~decoded).sum())
    widths = [4, 8, 16, 24, n_und]
    r = observation2(m, x_prev, x, decoded, widths, n_active=4)
    assert r["W"] == widths and len(r["active"]) == 4
    assert all(v >= 0 for v in r["truncation"] + r["truncation_cache"])
    # the whole undecoded context visible: truncation is the reference itself
    assert r["truncation"][-1] == 0.0
    # W = |A|: no buffer token, so caching changes nothing
    assert r["truncation_cache"][0] == r["truncation"][0]
    # with caching, a buffer that did not change since t0 - 1 only differs
    # through the rows decoded at t0 - 1 (their tokens feed the cached K/V)
    assert r["truncation_cache"][-1] > 0.0
    print("Observation 2 probe (random weights):", r)


def test_probe_subset_forward_equals_plain_forward():
    shape = synth.ModelShape(n_layers=2, hidden=32, n_heads=2, n_kv_heads=1, head_dim=16,
                             ffn=48, vocab=40, dtype=synth.DTYPE_F32)
    m = OracleModel(synth.Weights(shape, seed=1, std=0.3))
    x = np.array([1, 5, 9, 2, 39, 39, 7, 39], dtype=np.int64)
    h1, K1, _ = _forward_subset(m, x, list(range(len(x))))
    h2, K2, _ = m.forward(x)
    np.testing.assert_array_equal(h1, h2)
    np.testing.assert_array_equal(K1[1], K2[1])
    # keeping rows with their own K/V reproduces the plain forward
    h3, _, _ = _forward_subset(m, x, list(range(len(x))), {"K": K2, "V": m.forward(x)[2]},
                               keep=[4, 5])
    np.testing.assert_allclose(h3, h2, rtol=0, atol=1e-13)
    p = np.array([[0.5, 0.5, 0.0]])
    assert kl_rows(p, p)[0] == 0.0 and kl_rows(p, np.array([[0.25, 0.5, 0.25]]))[0] > 0


# ---- the truncation + cache leg, pinned against an independent loop model ----

def _loop_subset(lm, ids, rows, kept=None):
    """Loop-model forward over the visible positions `rows` (absolute
    positions, every row attends to every visible row).  `kept` maps a
    position to its per-layer (K, V), which replace the computed ones at that
    position.  Returns ({position: h}, [{position: (K, V)} per layer])."""
    hs = {p: list(lm.t["emb"][int(ids[p])]) for p in rows}
    kv_layers = []
    for l in range(lm.s.n_layers):
        per = {p: lm.qkv(l, hs[p], p) for p in rows}
        kv = {p: (per[p][1], per[p][2]) for p in rows}
        if kept:
            for p, layers in kept.items():
                kv[p] = layers[l]
        kv_layers.append(kv)
        Ks = [kv[p][0] for p in rows]
        Vs = [kv[p][1] for p in rows]
        hs = {p: lm.rest(l, hs[p], lm.attend(per[p][0], Ks, Vs)) for p in rows}
    return hs, kv_layers


def _loop_probs(lm, h, mask_id):
    """Predictive distribution of one row, [MASK] excluded, by explicit loops."""
    import math
    lg = lm.logits(h)
    mx = max(v for i, v in enumerate(lg) if i != mask_id)
    e = [0.0 if i == mask_id else math.exp(v - mx) for i, v in enumerate(lg)]
    tot = sum(e)
    return [v / tot for v in e]


def _loop_kl(p, q):
    import math
    return sum(a * (math.log(a) - math.log(b)) for a, b in zip(p, q) if a > 0)


def _micro():
    from test_oracle_bruteforce import LoopModel, micro_shape
    shape = micro_shape(synth.DTYPE_F32, True, 2)
    W = synth.Weights(shape, seed=21, std=0.25)
    return OracleModel(W), LoopModel(W), shape


def test_subset_forward_keeps_cached_rows_at_their_positions():
    """Visible rows with holes (positions != indices) and kept rows whose K/V
    come from a different token state: the oracle must place every kept
    row's cached K/V at that row's own position."""
    om, lm, shape = _micro()
    rng = np.random.default_rng(8)
    x_prev = rng.integers(0, shape.vocab - 1, size=16)
    x = x_prev.copy()
    x[[2, 9, 12]] = rng.integers(0, shape.vocab - 1, size=3)   # tokens that changed
    rows = [0, 1, 2, 5, 6, 9, 11, 12, 14]
    keep = [6, 11, 14]                                           # all after a hole
    _, Kp, Vp = _forward_subset(om, x_prev, rows)
    h, _, _ = _forward_subset(om, x, rows, {"K": Kp, "V": Vp}, keep=keep)
    _, kv_prev = _loop_subset(lm, x_prev, rows)
    kept = {p: [kv_prev[l][p] for l in range(shape.n_layers)] for p in keep}
    hb, _ = _loop_subset(lm, x, rows, kept)
    np.testing.assert_allclose(h, np.array([hb[p] for p in rows]), rtol=1e-12, atol=1e-12)
    # the kept K/V matter: without them the result differs
    h_fresh, _, _ = _forward_subset(om, x, rows)
    assert np.abs(h_fresh - h).max() > 1e-6


def test_observation2_equals_loop_model_computation():
    """Both KL curves of the probe recomputed independently with the loop
    model: the reference from a forward over every position, truncation from
    a forward over the visible positions, truncation + cache with the buffer
    rows' K/V taken from the state of step t0 - 1 over the same positions."""
    om, lm, shape = _micro()
    prompt = [3, 14, 15, 9, 26]
    G = 18
    x_prev, x, decoded = _state(om, prompt, G, t0=4)
    assert (x_prev != x).any()
    n_act = 3
    und = [int(i) for i in np.flatnonzero(~decoded)]
    dec = [int(i) for i in np.flatnonzero(decoded)]
    A = und[:n_act]
    widths = [3, 5, 8, len(und)]
    r = observation2(om, x_prev, x, decoded, widths, n_active=n_act)
    assert r["active"] == A and r["W"] == widths
    mask = shape.mask_id
    h_ref, _ = _loop_subset(lm, x, list(range(len(x))))
    ref = [_loop_probs(lm, h_ref[p], mask) for p in A]
    for i, W in enumerate(widths):
        rows = sorted(dec + und[:W])
        h_t, _ = _loop_subset(lm, x, rows)
        kl_t = sum(_loop_kl(ref[a], _loop_probs(lm, h_t[p], mask)) for a, p in enumerate(A)) / n_act
        _, kv_prev = _loop_subset(lm, x_prev, rows)
        buffer = [p for p in und[:W] if p not in A]
        kept = {p: [kv_prev[l][p] for l in range(shape.n_layers)] for p in buffer}
        h_c, _ = _loop_subset(lm, x, rows, kept)
        kl_c = sum(_loop_kl(ref[a], _loop_probs(lm, h_c[p], mask)) for a, p in enumerate(A)) / n_act
        np.testing.assert_allclose(r["truncation"][i], kl_t, rtol=1e-9, atol=1e-14)
        np.testing.assert_allclose(r["truncation_cache"][i], kl_c, rtol=1e-9, atol=1e-14)
        if buffer:
            # sensitive to where the cached K/V come from: x_prev differs from x
            # at the positions decoded at t0 - 1, which reach the buffer rows'
            # K/V from the second layer on
            assert abs(kl_c - kl_t) > 1e-9 * max(kl_t, 1e-12), (W, kl_c, kl_t)


def test_cache_from_the_same_state_is_truncation_exactly():
    """With x_prev == x the cached K/V are the ones the truncated forward
    computes itself, so both curves agree exactly at every width."""
    om, _, shape = _micro()
    prompt = [3, 14, 15, 9, 26]
    _, x, decoded = _state(om, prompt, 18, t0=4)
    n_und = int((~decoded).sum())
    widths = [3, 4, 6, 9, n_und]
    r = observation2(om, x, x, decoded, widths, n_active=3)
    assert r["truncation_cache"] == r["truncation"]
    assert r["truncation"][-1] == 0.0 and r["truncation"][0] > 0.0
