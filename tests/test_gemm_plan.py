"""Host logic of the projection GEMM planner (no GPU): every plan it returns
for the projection shapes of the workloads and for a seeded sweep of other
widths is one its launchers accept, covers the product exactly once, and
keeps the limits its kernels assume."""
import numpy as np
import pytest

import synth

wd = pytest.importorskip("paper_2601_20332_amd")


def _shapes(model):
    """(N, K) of the four projections of a model (gate and up as one GEMM)."""
    H, d = model.hidden, model.head_dim
    qkv = (model.n_heads + 2 * model.n_kv_heads) * d
    return [(qkv, H), (H, model.n_heads * d), (2 * model.ffn, H), (H, model.ffn)]


WORKLOAD_SHAPES = sorted({s for w in synth.WORKLOADS.values() if w.model.dtype == synth.DTYPE_BF16
                          for s in _shapes(w.model)})
ROWS = [1, 2, 15, 16, 17, 33, 34, 39, 48, 63, 64, 65, 66, 80, 94, 96, 97, 127, 128, 129, 191,
        192, 224, 256, 257, 264, 320, 383, 384, 385, 528, 624, 768, 1024, 1536, 4096, 8000,
        16000]


def _check(M, N, K, fp8, max_splits=1 << 20):
    p = wd.wd_debug_gemm_plan(M, N, K, fp8, max_splits)
    where = f"M={M} N={N} K={K} fp8={fp8} max_splits={max_splits}: {p}"
    KT = K // 32
    assert p["accepted"] & 1, where
    assert 1 <= p["splits"] <= max_splits, where
    if p["kernel"] in (1, 2):  # powers of two up to 8
        assert p["splits"] in (1, 2, 4, 8), where
    ks = p["k_steps_per_split"]
    assert ks * p["splits"] >= KT and ks * (p["splits"] - 1) < KT, where
    assert N % p["features"] == 0, where
    tiles = -(-M // p["rows"]) * (N // p["features"])
    assert p["workgroups"] == tiles * p["splits"], where
    if p["kernel"] == 1:  # pipelined few-row kernel: every row in one tile
        assert M <= 96 and p["rows"] >= M and p["waves"] in (2, 3, 4, 6, 7), where
    elif p["kernel"] == 2:  # many-row kernel: bf16 weights only
        assert not fp8 and M > 64 and p["features"] in (256, 192, 128), where
        if p["waves"] == 4:  # several rounds of 256 x 256 tiles: one wave per SIMD
            assert (p["rows"], p["features"]) == (256, 256) and p["workgroups"] > 512, where
        else:
            assert p["waves"] == (12 if p["features"] == 192 else 8), where
        if p["features"] < 256:  # narrower tiles only within two rounds
            assert p["workgroups"] <= 512, where
        # the step loop applies SwiGLU in this kernel whenever K is not split
        assert bool(p["accepted"] & 2) == (p["splits"] == 1), where
    else:
        assert p["kernel"] == 3 and p["waves"] == 4, where
        assert not p["accepted"] & 2, where
    if fp8:
        assert K % 64 or ks % 2 == 0, where
    return p


@pytest.mark.parametrize("N,K", WORKLOAD_SHAPES)
def test_workload_projection_plans(N, K):
    for M in ROWS:
        for fp8 in (False, True):
            if fp8 and K % 64:
                continue
            _check(M, N, K, fp8)


def test_seeded_width_sweep():
    rng = np.random.default_rng(20601)
    for _ in range(400):
        N = int(rng.integers(1, 64)) * 64
        K = int(rng.integers(1, 200)) * 32
        M = int(rng.choice(ROWS))
        fp8 = bool(rng.integers(0, 2)) and K % 64 == 0
        _check(M, N, K, fp8, int(rng.choice([1, 2, 8, 1 << 20])))


def test_llada_refresh_rows_take_the_measured_tiles():
    # Q/K/V and gate/up at 264-384 rows: 192-row x 192-feature tiles, one
    # round of 256 workgroups; gate/up unsplit (SwiGLU in the epilogue)
    for M in (264, 320, 384):
        qkv = _check(M, 12288, 4096, False)
        gu = _check(M, 24576, 4096, False)
        assert (qkv["rows"], qkv["features"], qkv["splits"], qkv["workgroups"]) == (192, 192, 2, 256)
        assert (gu["rows"], gu["features"], gu["splits"], gu["workgroups"]) == (192, 192, 1, 256)
    # O at refresh rows: 128-feature tiles with 4 splits of 32 K steps
    o = _check(384, 4096, 4096, False)
    assert (o["features"], o["splits"], o["k_steps_per_split"]) == (128, 4, 32)
    # normal-step rows go to the pipelined few-row kernel for O and down
    assert _check(34, 4096, 4096, False)["kernel"] == 1
    assert _check(34, 4096, 12288, False)["kernel"] == 1


def test_batched_refresh_rows_take_pinned_256_tiles():
    # four or more rounds of unsplit 256 x 256 tiles: those tiles on the
    # pinned 4-wave schedule, whatever the work count prefers
    for M in (3000, 5000, 7000, 11000):
        gu = _check(M, 24576, 4096, False)
        assert (gu["rows"], gu["features"], gu["waves"], gu["splits"]) == (256, 256, 4, 1)
    for M in (7000, 9000, 14000):
        qkv = _check(M, 12288, 4096, False)
        assert (qkv["rows"], qkv["features"], qkv["waves"], qkv["splits"]) == (256, 256, 4, 1)
    # below four rounds the work count decides (Q/K/V at 3000 rows: 576 workgroups)
    assert _check(3000, 12288, 4096, False)["waves"] != 4


def test_narrow_products_take_the_pipelined_split_kernel():
    # Q/K/V of Dream-7B (4608 x 3584) is too narrow for the fused epilogue
    # kernel: up to 64 rows it runs the pipelined split kernel with 3 groups per
    # workgroup and 2 splits (so the Q/K/V epilogue reads 2 partials)
    for M in (34, 40, 46, 64):
        p = _check(M, 4608, 3584, False)
        assert (p["kernel"], p["waves"], p["splits"]) == (1, 3, 2), p
    # above 64 rows the many-row tiles keep it
    assert _check(80, 4608, 3584, False)["kernel"] == 2
    # wide products keep their plans (LLaDA-8B Q/K/V at normal-step rows is fused,
    # not planned here; O and down stay on 4 groups per workgroup)
    assert _check(39, 4096, 4096, False)["waves"] == 4


def test_invalid_arguments():
    with pytest.raises(wd.WdError):
        wd.wd_debug_gemm_plan(0, 256, 256)
    with pytest.raises(wd.WdError):
        wd.wd_debug_gemm_plan(16, 256, 48)
    with pytest.raises(wd.WdError):
        wd.wd_debug_gemm_plan(1 << 25, 256, 256)
