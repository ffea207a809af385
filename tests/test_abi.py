"""The C ABI without a GPU: the library loads, exports every function the
header declares, its host-side schedule matches the oracle's bit for bit, and
invalid arguments are rejected before any device work."""
import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import synth
from oracle.schedule import plan_counts

wd = pytest.importorskip("paper_2601_20332_amd")

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "wd.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wd_[a-z_]+)\s*\(", text)))


def test_every_declared_function_is_exported():
    names = header_functions()
    assert len(names) >= 17
    for n in names:
        assert hasattr(wd.lib, n), n
    assert sorted(wd.EXPORTED) == names


def cfg_of(shape: synth.ModelShape):
    return wd.model_config(n_layers=shape.n_layers, hidden=shape.hidden, n_heads=shape.n_heads,
                           n_kv_heads=shape.n_kv_heads, head_dim=shape.head_dim, ffn=shape.ffn,
                           vocab=shape.vocab, mask_id=shape.mask_id, dtype=shape.dtype,
                           qkv_bias=shape.qkv_bias, rms_eps=shape.rms_eps,
                           rope_theta=shape.rope_theta)


@pytest.mark.parametrize("name", ["tiny", "llada8b", "dream7b"])
def test_weight_inventory_matches_generator(name):
    shape = synth.WORKLOADS[name].model
    cfg = cfg_of(shape)
    specs = synth.tensor_specs(shape)
    assert wd.wd_weight_count(cfg) == len(specs)
    for i, (_, shp, _) in enumerate(specs):
        r, c = wd.wd_weight_shape(cfg, i)
        assert (r, c) == (shp[0], shp[1] if len(shp) > 1 else 1)
    esz = 2 if shape.dtype == synth.DTYPE_BF16 else 4
    n_params = sum(int(np.prod(s)) for _, s, _ in specs)
    assert n_params * esz <= wd.wd_model_bytes(cfg) <= n_params * esz + 256 * len(specs)


def test_unsupported_configs_rejected():
    base = dict(n_layers=2, hidden=256, n_heads=2, n_kv_heads=2, head_dim=128, ffn=512, vocab=1024,
                mask_id=1023, dtype="bf16", qkv_bias=0, rms_eps=1e-5, rope_theta=1e4)
    assert wd.wd_weight_count(wd.model_config(**base)) > 0
    for bad in [dict(head_dim=96), dict(n_kv_heads=3), dict(hidden=200), dict(mask_id=1024),
                dict(vocab=1000, mask_id=999), dict(rms_eps=0.0), dict(n_layers=0),
                dict(dtype="bf16", head_dim=64)]:
        c = wd.model_config(**{**base, **bad})
        assert wd.wd_weight_count(c) == -1
        assert wd.wd_model_bytes(c) == 0


def test_init_rejects_bad_arguments_without_touching_the_device():
    cfg = wd.model_config(n_layers=1, hidden=256, n_heads=2, n_kv_heads=2, head_dim=128, ffn=512,
                          vocab=1024, mask_id=1023, dtype="bf16", qkv_bias=0, rms_eps=1e-5,
                          rope_theta=1e4)
    h = ctypes.c_void_p()
    n = wd.wd_weight_count(cfg)
    ptrs = (ctypes.c_void_p * n)(*([256] * n))
    st = wd.lib.wd_init_model(ctypes.byref(cfg), ptrs, n - 1, ctypes.c_void_p(256), 1 << 30, None,
                              ctypes.byref(h))
    assert st == wd.WD_ERR_INVALID_ARG and "weight pointers" in wd.wd_last_error()
    ptrs[3] = 0
    st = wd.lib.wd_init_model(ctypes.byref(cfg), ptrs, n, ctypes.c_void_p(256), 1 << 30, None,
                              ctypes.byref(h))
    assert st == wd.WD_ERR_INVALID_ARG and "NULL" in wd.wd_last_error()
    ptrs[3] = 264
    st = wd.lib.wd_init_model(ctypes.byref(cfg), ptrs, n, ctypes.c_void_p(256), 1 << 30, None,
                              ctypes.byref(h))
    assert st == wd.WD_ERR_INVALID_ARG and "aligned" in wd.wd_last_error()
    ptrs[3] = 256
    st = wd.lib.wd_init_model(ctypes.byref(cfg), ptrs, n, ctypes.c_void_p(256), 16, None,
                              ctypes.byref(h))
    assert st == wd.WD_ERR_OUT_OF_MEMORY
    assert h.value is None


def test_null_handles_rejected():
    for f in (wd.lib.wd_step, wd.lib.wd_full_step):
        assert f(None, None) == wd.WD_ERR_INVALID_ARG
    assert wd.lib.wd_slide_window(None) == wd.WD_ERR_INVALID_ARG
    assert wd.lib.wd_refresh_buffer(None) == wd.WD_ERR_INVALID_ARG
    wd.lib.wd_free_seq(None)
    wd.lib.wd_free_model(None)
    lens = np.array([4], np.int32)
    win = wd.window_config(2, 2, 2, 1)
    assert wd.lib.wd_seq_bytes(None, ctypes.byref(win), 1, wd._i32p(lens), 8) == 0


def test_plan_rejects_bad_windows():
    for w in [(0, 2, 2, 1), (2, -1, 2, 1), (2, 2, 0, 1), (2, 2, 2, 0), (65, 0, 1, 1)]:
        with pytest.raises(wd.WdError):
            wd.wd_plan(4, 8, wd.window_config(*w))
    with pytest.raises(wd.WdError):
        wd.wd_plan(4, 0, wd.window_config(2, 2, 2, 1))


def _compare_plan(n_p, G, win, refresh="full"):
    ref = plan_counts(n_p, G, win, refresh=refresh)
    got = wd.wd_plan(n_p, G, wd.window_config(win.n_active, win.n_buffer, win.refresh_every,
                                              win.unmask_per_step,
                                              buffer_refresh=refresh == "buffer"))
    assert len(got["n_rows"]) == len(ref)
    assert got["is_refresh"].tolist() == [int(p.refresh) for p in ref]
    assert got["ctx_len"].tolist() == [p.ctx_len for p in ref]
    assert got["n_active"].tolist() == [p.n_active for p in ref]
    assert got["n_rows"].tolist() == [p.n_online for p in ref]
    assert got["n_decode"].tolist() == [p.n_decode for p in ref]


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_plan_matches_oracle_on_workloads(name):
    w = synth.WORKLOADS[name]
    for n_p in sorted({w.prompt_len, *(w.ragged_prompt or ())}):
        _compare_plan(n_p, w.gen_len, w.window)


@settings(max_examples=300, deadline=None)
@given(n_p=st.integers(0, 40), G=st.integers(1, 200), na=st.integers(1, 64),
       nb=st.integers(0, 70), R=st.integers(1, 20), k=st.integers(1, 8))
def test_plan_matches_oracle_everywhere(n_p, G, na, nb, R, k):
    _compare_plan(n_p, G, synth.WindowSettings(na, nb, R, k))
    _compare_plan(n_p, G, synth.WindowSettings(na, nb, R, k), refresh="buffer")


def test_plan_rejects_bad_variant_flags():
    for field in ("stop_at_eos", "buffer_refresh"):
        win = wd.window_config(2, 2, 2, 1)
        setattr(win, field, 2)
        with pytest.raises(wd.WdError):
            wd.wd_plan(4, 8, win)
