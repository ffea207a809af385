"""Pins of the oracle's building blocks against library routines, closed
forms and hand-checked values."""
import math

import numpy as np
import pytest
import scipy.special
import torch

import synth
from oracle import numerics as nm
from oracle.sampler import confidence, select_updates, top1_margin


# -- bf16 rounding ------------------------------------------------------------

def test_round_bf16_matches_torch_on_float32_inputs():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(200000).astype(np.float32) * 3,
                        rng.standard_normal(1000).astype(np.float32) * 1e-30,
                        rng.standard_normal(1000).astype(np.float32) * 1e30])
    # values exactly halfway between two bf16 neighbours
    base = synth.bf16_bits_to_f32(rng.integers(0x3000, 0x5000, 4000).astype(np.uint16))
    ties = (base.view(np.uint32) | np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(nm.round_bf16(x.astype(np.float64)), ref)


def test_round_bf16_hand_values():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even significand (1)
    assert nm.round_bf16(1.0 + 2.0 ** -8) == 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 (odd) and 1 + 2^-6 (even)
    assert nm.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6
    assert nm.round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -30) == 1.0 + 2.0 ** -7
    assert nm.round_bf16(-3.0) == -3.0
    assert nm.round_bf16(0.0) == 0.0
    assert nm.round_bf16(255.5) == 256.0     # 8 significant bits: 255.5 -> tie -> 256


def test_storage_conversion_is_torch_rne():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(100000).astype(np.float32)
    bits = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(bits, ref)


# -- RMSNorm -------------------------------------------------------------------

def test_rmsnorm_matches_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((7, 64)) * 3
    g = rng.standard_normal(64)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (64,), torch.from_numpy(g),
                                       eps=1e-5).numpy()
    np.testing.assert_allclose(nm.rmsnorm(x, g, 1e-5), ref, rtol=1e-12, atol=1e-13)


def test_rmsnorm_unit_rms():
    x = np.random.default_rng(3).standard_normal((4, 128))
    y = nm.rmsnorm(x, np.ones(128), 0.0)
    np.testing.assert_allclose(np.sqrt((y * y).mean(-1)), 1.0, rtol=1e-12)


# -- RoPE ----------------------------------------------------------------------

def test_rope_as_complex_rotation():
    """Pair (i, i + d/2) as the complex number x_i + j x_{i+d/2}; RoPE multiplies
    it by exp(j * pos * theta^(-2i/d))."""
    rng = np.random.default_rng(4)
    d, theta = 16, 500000.0
    x = rng.standard_normal((5, 3, d))
    pos = np.array([0, 1, 7, 100, 1535])
    z = x[..., :d // 2] + 1j * x[..., d // 2:]
    ang = pos[:, None] * theta ** (-np.arange(0, d, 2) / d)[None, :]
    zr = z * np.exp(1j * ang)[:, None, :]
    ref = np.concatenate([zr.real, zr.imag], axis=-1)
    np.testing.assert_allclose(nm.apply_rope(x, pos, theta), ref, rtol=1e-12, atol=1e-12)


def test_rope_hand_value_and_invariants():
    # d = 2: one pair, angle = pos radians; (1, 0) at pos 1 -> (cos 1, sin 1)
    y = nm.apply_rope(np.array([[[1.0, 0.0]]]), np.array([1]), 10000.0)
    np.testing.assert_allclose(y[0, 0], [math.cos(1.0), math.sin(1.0)], rtol=1e-15)
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 1, 64))
    k = rng.standard_normal((1, 1, 64))
    # position 0 is the identity; norms are preserved
    np.testing.assert_allclose(nm.apply_rope(q, [0], 1e4), q, rtol=0, atol=0)
    qr = nm.apply_rope(q, [37], 1e4)
    assert abs(np.linalg.norm(qr) - np.linalg.norm(q)) < 1e-12
    # q(m).k(n) depends only on m - n
    a = (nm.apply_rope(q, [10], 1e4) * nm.apply_rope(k, [3], 1e4)).sum()
    b = (nm.apply_rope(q, [107], 1e4) * nm.apply_rope(k, [100], 1e4)).sum()
    c = (nm.apply_rope(q, [3], 1e4) * nm.apply_rope(k, [10], 1e4)).sum()
    assert abs(a - b) < 1e-12
    assert abs(a - c) > 1e-6


# -- attention -----------------------------------------------------------------

@pytest.mark.parametrize("nh,nkv", [(4, 4), (8, 2), (28, 4)])
def test_attention_matches_torch_sdpa(nh, nkv):
    rng = np.random.default_rng(6)
    nq, nk, d = 5, 11, 16
    q = rng.standard_normal((nq, nh, d))
    k = rng.standard_normal((nk, nkv, d))
    v = rng.standard_normal((nk, nkv, d))
    valid = rng.random(nk) > 0.3
    valid[0] = True
    tq = torch.from_numpy(q).permute(1, 0, 2)
    tk = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(nh // nkv, dim=0)
    tv = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(nh // nkv, dim=0)
    mask = torch.from_numpy(valid)[None, None, :].expand(nh, nq, nk)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask,
                                                           is_causal=False)
    ref = ref.permute(1, 0, 2).numpy()
    np.testing.assert_allclose(nm.attention(q, k, v, valid), ref, rtol=1e-12, atol=1e-12)


def test_attention_identical_keys_average_values():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((3, 2, 8))
    k = np.repeat(rng.standard_normal((1, 2, 8)), 6, axis=0)
    v = rng.standard_normal((6, 2, 8))
    np.testing.assert_allclose(nm.attention(q, k, v), np.broadcast_to(v.mean(0), (3, 2, 8)),
                               rtol=1e-12, atol=1e-12)


def test_silu_matches_torch():
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(nm.silu(z), torch.nn.functional.silu(torch.from_numpy(z)).numpy(),
                               rtol=1e-13, atol=1e-300)


# -- confidence and selection -----------------------------------------------------

def test_confidence_is_max_softmax_probability_without_mask():
    rng = np.random.default_rng(8)
    V, mask = 300, 299
    l = rng.standard_normal((6, V)) * 2
    l[2, mask] = 50.0                    # a huge [MASK] logit must be ignored
    tok, conf = confidence(l, mask)
    ref = l.copy()
    ref[:, mask] = -np.inf
    p = scipy.special.softmax(ref, axis=1)
    np.testing.assert_array_equal(tok, p.argmax(1))
    np.testing.assert_allclose(conf, p.max(1).astype(np.float32), rtol=1e-6)
    np.testing.assert_allclose(p.sum(1), 1.0, rtol=1e-12)


def test_confidence_ties_take_lowest_id():
    l = np.zeros((2, 10))
    l[0, [3, 7]] = 1.0
    l[1, [9, 4]] = 2.0
    l[1, 0] = 2.0
    tok, conf = confidence(l, 0)          # id 0 is the mask: excluded even at the max
    assert tok.tolist() == [3, 4]
    np.testing.assert_allclose(conf[0], 1.0 / (2 + 7 * math.exp(-1.0)), rtol=1e-6)


def test_select_updates_ties_lowest_position():
    assert select_updates([5, 9, 2, 7], [0.5, 0.9, 0.5, 0.9], 3) == [7, 9, 2]
    assert select_updates([4], [0.1], 2) == [4]
    assert select_updates([], [], 2) == []


def test_top1_margin():
    l = np.array([[1.0, 3.0, 2.5, 9.0]])
    assert top1_margin(l, 3)[0] == pytest.approx(0.5)
