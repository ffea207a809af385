"""The FP8-weight variant (not the paper's precision) on the GPU: the
library's packed e4m3 codes and row scales equal the oracle quantizer's
exactly (and bf16 packing keeps every weight), and whole generations match
the oracle's FP8 model step by step.  Runs on an MI355X only."""
import numpy as np
import pytest

import synth
from oracle.model import OracleModel
from oracle.quant import e4m3_value, quantize_rows
from wdtest import check_sequence, gpu_model, log, run_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)
import paper_2601_20332_amd as wd  # noqa: E402

MICRO_GQA = synth.ModelShape(n_layers=3, hidden=512, n_heads=4, n_kv_heads=2, head_dim=128,
                             ffn=1024, vocab=2048, dtype=synth.DTYPE_BF16, qkv_bias=True,
                             rms_eps=1e-6, rope_theta=1e6)
MATRICES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd", "lm_head")


def _rows_to_check(n):
    return sorted({0, 1, 7, 8, 63, 64, 65, n // 2, n - 9, n - 1})


@pytest.mark.parametrize("fp8", [False, True], ids=["bf16", "fp8"])
def test_packed_weights_exact(fp8):
    W = synth.Weights(MICRO_GQA, seed=11)
    m = gpu_model(W, weight_fp8=fp8)
    specs = synth.tensor_specs(MICRO_GQA)
    checked = 0
    for idx, (name, shape, _) in enumerate(specs):
        leaf = name.split(".")[-1]
        if leaf not in MATRICES or (name.startswith("layers.") and not name.startswith("layers.1.")
                                    and leaf != "lm_head"):
            continue
        w = W.f32(name)
        if fp8:
            codes, scales = quantize_rows(w)
        for r in _rows_to_check(shape[0]):
            vals, sc = wd.wd_debug_weight_row(m, idx, r, shape[1])
            if fp8:
                np.testing.assert_array_equal(vals, e4m3_value(codes[r]).astype(np.float32),
                                              err_msg=f"{name} row {r}")
                assert sc == scales[r], (name, r, sc, scales[r])
            else:
                np.testing.assert_array_equal(vals, w[r], err_msg=f"{name} row {r}")
                assert sc == 1.0
            checked += 1
    assert checked > 60
    m.free()


def _parity(shape, prompts, G, win, seed=0, max_steps=None):
    log(f"[case] fp8 {shape} prompts={[len(p) for p in prompts]} G={G} win={win}")
    W = synth.Weights(shape, seed=seed)
    m = gpu_model(W, weight_fp8=True)
    steps, _ = run_gpu(m, prompts, G, win, max_steps=max_steps)
    m.free()
    om = OracleModel(W, weight_format="fp8")
    for b, p in enumerate(prompts):
        rep = check_sequence(om, p, G, win, steps, b, len(prompts), max_steps=max_steps)
        print(f"PARITY-FP8 L={shape.n_layers} H={shape.hidden} seq={b} steps={rep.steps} "
              f"max_rel_logit_err={rep.max_rel:.3e} adopted_sel={rep.select_adopted} "
              f"adopted_tok={rep.token_adopted}", flush=True)
        assert rep.steps == len(steps)


def test_fp8_gqa_bias_batched():
    _parity(MICRO_GQA, synth.prompts(MICRO_GQA, [33, 50]), 24, synth.WindowSettings(5, 7, 4, 2))


def test_fp8_llada_shape_two_layers():
    """Full-width LLaDA-8B layers (the fused Q/K/V and SwiGLU kernels, the
    126464-row LM head) with fp8 weights, first 10 steps."""
    w = synth.WORKLOADS["llada8b"]
    shape = synth.with_layers(w.model, 2)
    _parity(shape, synth.prompts(shape, [w.prompt_len]), w.gen_len, w.window, max_steps=10)


def test_fp8_needs_a_bf16_model():
    shape = synth.WORKLOADS["tiny"].model
    with pytest.raises(wd.WdError) as e:
        gpu_model(synth.Weights(shape), weight_fp8=True)
    assert e.value.status in (wd.WD_ERR_UNSUPPORTED, wd.WD_ERR_INVALID_ARG)
