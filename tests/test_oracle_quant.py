"""Pins of the oracle's e4m3 quantizer (the FP8-weight variant): codes
derived by hand from the format definition, a round trip over every finite
code, agreement with an independent converter (torch.float8_e4m3fn) on
random values, and the rounding error bound."""
import numpy as np
import pytest

from oracle.quant import (E4M3_MAX, dequantize_rows, e4m3_encode, e4m3_value,
                          quantize_rows)

# value -> code, by hand: code = sign<<7 | E<<3 | M, value = 2^(E-7) (1 + M/8),
# E = 0: M * 2^-9; ties go to the even mantissa
HAND = [
    (1.0, 0x38),             # E = 7, M = 0
    (448.0, 0x7E),           # largest finite: E = 15, M = 6
    (500.0, 0x7E),           # saturates
    (2.0 ** -9, 0x01),       # smallest subnormal
    (0.1, 0x1D),             # 0.1015625 = 2^-4 * 1.625
    (300.0, 0x79),           # nearest 288 = 2^8 * 1.125
    (17.0, 0x58),            # tie 16 | 18 -> 16 (even mantissa)
    (19.0, 0x5A),            # tie 18 | 20 -> 20
    (2.0 ** -10, 0x00),      # tie 0 | 2^-9 -> 0
    (3 * 2.0 ** -10, 0x02),  # tie 2^-9 | 2^-8 -> 2^-8
    (0.0, 0x00),
    (-1.5, 0xBC),            # sign, E = 7, M = 4
    (2.0 ** -6, 0x08),       # smallest normal
    (15 * 2.0 ** -10, 0x08), # tie 7*2^-9 | 2^-6 -> 2^-6 (code 8 is even)
]


@pytest.mark.parametrize("value,code", HAND)
def test_hand_codes(value, code):
    assert int(e4m3_encode(np.float32(value))) == code


def test_every_finite_code_round_trips():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    np.testing.assert_array_equal(e4m3_encode(e4m3_value(codes).astype(np.float32)), codes)
    assert e4m3_value(0x7E) == 448.0 and e4m3_value(0x01) == 2.0 ** -9


def test_matches_an_independent_converter():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.uniform(-E4M3_MAX, E4M3_MAX, 50000),
                        rng.normal(0, 1e-2, 50000),
                        rng.normal(0, 1.0, 50000)]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(e4m3_encode(x), ref)


def test_rounding_error_bound_and_scales():
    rng = np.random.default_rng(1)
    w = (rng.normal(0, 0.02, (37, 300))).astype(np.float32)
    w[3] = 0.0
    codes, scale = quantize_rows(w)
    assert scale[3] == 1.0 and not codes[3].any()
    np.testing.assert_allclose(scale[:3], np.abs(w[:3]).max(axis=1) / np.float32(448), rtol=1e-7)
    # each row's largest magnitude maps to 448 (0x7E)
    assert ((codes[[0, 1, 2, 4]] & 0x7F) == 0x7E).any(axis=1).all()
    d = dequantize_rows(codes, scale)
    a = np.abs(w.astype(np.float64) / scale[:, None])
    # half a unit in the last place: 2^-4 relative for normals, 2^-10 absolute below 2^-6
    bound = np.where(a >= 2.0 ** -6, a * 2.0 ** -4, 2.0 ** -10) * scale[:, None]
    assert (np.abs(d - w) <= bound + 1e-12).all()


def test_fp8_model_quantizes_only_the_projection_matrices():
    import synth
    from oracle.model import OracleModel
    shape = synth.ModelShape(n_layers=1, hidden=64, n_heads=1, n_kv_heads=1, head_dim=64,
                             ffn=128, vocab=96, dtype=synth.DTYPE_BF16, qkv_bias=True)
    W = synth.Weights(shape, seed=5)
    plain, q8 = OracleModel(W), OracleModel(W, weight_format="fp8")
    for name in ("layers.0.wq", "layers.0.wo", "layers.0.wd", "lm_head"):
        np.testing.assert_array_equal(q8.w(name), dequantize_rows(*quantize_rows(W.f32(name))))
        assert not np.array_equal(q8.w(name), plain.w(name))
    for name in ("layers.0.attn_norm", "layers.0.bq", "final_norm"):
        np.testing.assert_array_equal(q8.w(name), plain.w(name))
    np.testing.assert_array_equal(q8.emb_rows([1, 2]), plain.emb_rows([1, 2]))
    with pytest.raises(ValueError):
        OracleModel(synth.Weights(synth.WORKLOADS["tiny"].model), weight_format="fp8")
