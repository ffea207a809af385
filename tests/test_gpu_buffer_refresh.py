"""GPU parity of the buffer-only refresh variant (not the paper's method:
later refreshes recompute only the window and the previous phase's decoded
positions) against the oracle's variant, step by step.  Runs on an MI355X
only."""
import numpy as np
import pytest

import synth
from oracle.model import OracleModel
from wdtest import check_sequence, gpu_model, log, run_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)
import paper_2601_20332_amd as wd  # noqa: E402

MICRO_GQA = synth.ModelShape(n_layers=3, hidden=512, n_heads=4, n_kv_heads=2, head_dim=128,
                             ffn=1024, vocab=2048, dtype=synth.DTYPE_BF16, qkv_bias=True,
                             rms_eps=1e-6, rope_theta=1e6)


def _run(shape, prompts, G, win, seed=0):
    log(f"[case] buffer refresh {shape.dtype} prompts={[len(p) for p in prompts]} G={G} win={win}")
    W = synth.Weights(shape, seed=seed)
    m = gpu_model(W)
    steps, _ = run_gpu(m, prompts, G, win, refresh="buffer")
    m.free()
    om = OracleModel(W)
    for b, p in enumerate(prompts):
        rep = check_sequence(om, p, G, win, steps, b, len(prompts), refresh="buffer")
        print(f"PARITY-BUF {shape.dtype} seq={b} steps={rep.steps} "
              f"max_rel_logit_err={rep.max_rel:.3e} adopted_sel={rep.select_adopted} "
              f"adopted_tok={rep.token_adopted}", flush=True)
        assert rep.steps == len(steps)
        if shape.dtype == synth.DTYPE_F32:
            assert rep.token_adopted == 0 and rep.select_adopted == 0
    return steps


def test_buffer_refresh_tiny_fp32():
    w = synth.WORKLOADS["tiny"]
    steps = _run(w.model, synth.prompts(w.model, [w.prompt_len]), w.gen_len, w.window)
    plan = wd.wd_plan(w.prompt_len, w.gen_len,
                      wd.window_config(w.window.n_active, w.window.n_buffer,
                                       w.window.refresh_every, w.window.unmask_per_step,
                                       buffer_refresh=True))
    assert [s.res.n_rows for s in steps] == plan["n_rows"].tolist()
    # later refreshes run fewer rows than the retained prefix
    later = [i for i, r in enumerate(plan["is_refresh"]) if r][1:]
    assert later and all(plan["n_rows"][i] < plan["ctx_len"][i] for i in later)


def test_buffer_refresh_tiny_fp32_batch_ragged():
    shape = synth.WORKLOADS["tiny"].model
    _run(shape, synth.prompts(shape, [20, 33, 41]), 30, synth.WindowSettings(6, 8, 3, 2))


def test_buffer_refresh_bf16_gqa_batch():
    _run(MICRO_GQA, synth.prompts(MICRO_GQA, [33, 50]), 24, synth.WindowSettings(5, 7, 4, 2))


def test_buffer_refresh_with_eos_is_unsupported():
    shape = synth.WORKLOADS["tiny"].model
    m = gpu_model(synth.Weights(shape))
    wc = wd.window_config(4, 4, 2, 1, eos_id=3, buffer_refresh=True)
    with pytest.raises(wd.WdError) as e:
        wd.wd_prefill_prompt(m, synth.prompts(shape, [10]), 8, wc)
    assert e.value.status == wd.WD_ERR_UNSUPPORTED
    m.free()
