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
