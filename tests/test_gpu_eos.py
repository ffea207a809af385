"""GPU parity of adaptive termination at <eos> (Sec. 4.2): the HIP path
through the C ABI against the oracle's windowed and full decoders with the
same <eos> id, step by step, on seeded inputs.  The <eos> id of a case is a
token the oracle decodes at a chosen step without adaptive termination, so
that the cut happens by the model's own argmax on both sides.  Runs on an
MI355X only."""
import numpy as np
import pytest

import synth
from oracle.model import OracleModel
from oracle.schedule import FullDecoder, WindowedDecoder
from wdtest import check_sequence, gpu_model, log, run_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)
import paper_2601_20332_amd as wd  # noqa: E402

MICRO_GQA = synth.ModelShape(n_layers=3, hidden=512, n_heads=4, n_kv_heads=2, head_dim=128,
                             ffn=1024, vocab=2048, dtype=synth.DTYPE_BF16, qkv_bias=True,
                             rms_eps=1e-6, rope_theta=1e6)


def _token_decoded_at(om, prompt, G, win, step, full=False):
    """A token the oracle (no adaptive termination) decodes for the first time
    at `step` or soon after, so that as <eos> it ends the sequence there."""
    dec = (FullDecoder(om, prompt, G, win.unmask_per_step) if full
           else WindowedDecoder(om, prompt, G, win))
    seen = set()
    while not dec.done():
        rec = dec.step()
        new = [rec.chosen_tokens[p] for p in rec.selected if rec.chosen_tokens[p] not in seen]
        if rec.t >= step and new:
            return int(new[0])
        seen.update(rec.chosen_tokens.values())
    raise AssertionError("no fresh token after the chosen step")


def _run(shape, prompts, G, win, eos_from=(0, 3), full=False, seed=0):
    W = synth.Weights(shape, seed=seed)
    om = OracleModel(W)
    b0, step = eos_from
    eos = _token_decoded_at(om, prompts[b0], G, win, step, full=full)
    log(f"[case] {shape.dtype} prompts={[len(p) for p in prompts]} G={G} win={win} "
        f"full={full} eos={eos}")
    m = gpu_model(W)
    ends = []
    steps, final = run_gpu(m, prompts, G, win, full=full, eos_id=eos, ends=ends)
    m.free()
    reps = []
    for b, p in enumerate(prompts):
        rep = check_sequence(om, p, G, win, steps, b, len(prompts), full=full, eos_id=eos,
                             gpu_end=ends[b])
        print(f"PARITY-EOS {shape.dtype} seq={b} end={ends[b]}/{len(p) + G} steps={rep.steps} "
              f"max_rel_logit_err={rep.max_rel:.3e} adopted_sel={rep.select_adopted} "
              f"adopted_tok={rep.token_adopted}", flush=True)
        if shape.dtype == synth.DTYPE_F32:
            assert rep.token_adopted == 0 and rep.select_adopted == 0
        # nothing past the end was decoded after the end moved there: positions
        # past it that are undecoded keep the mask token
        tok, dec = final[0][b], final[1][b]
        assert dec[:ends[b]].all()
        assert (tok[ends[b]:][~dec[ends[b]:]] == shape.mask_id).all()
        reps.append(rep)
    assert ends[b0] < len(prompts[b0]) + G, "the chosen <eos> did not end its sequence"
    return steps, ends, reps


def test_eos_tiny_fp32_single():
    w = synth.WORKLOADS["tiny"]
    prompts = synth.prompts(w.model, [w.prompt_len])
    steps, ends, _ = _run(w.model, prompts, w.gen_len, w.window, eos_from=(0, 6))
    plain = len(wd.wd_plan(w.prompt_len, w.gen_len,
                           wd.window_config(*[getattr(w.window, f) for f in
                                              ("n_active", "n_buffer", "refresh_every",
                                               "unmask_per_step")]))["n_rows"])
    assert len(steps) < plain


def test_eos_tiny_fp32_batch_ragged():
    """Sequences end at different steps: per-sequence phase clocks, mixed
    refresh and normal rows in one step, finished sequences idle."""
    shape = synth.WORKLOADS["tiny"].model
    prompts = synth.prompts(shape, [20, 33, 41])
    _run(shape, prompts, 40, synth.WindowSettings(6, 8, 3, 2), eos_from=(1, 5))


def test_eos_bf16_gqa_batch():
    prompts = synth.prompts(MICRO_GQA, [33, 50])
    _run(MICRO_GQA, prompts, 24, synth.WindowSettings(5, 7, 4, 2), eos_from=(0, 4))


def test_eos_full_sequence_path():
    shape = synth.WORKLOADS["tiny"].model
    prompts = synth.prompts(shape, [24, 30])
    _run(shape, prompts, 20, synth.WindowSettings(4, 4, 2, 2), eos_from=(0, 2), full=True)


@pytest.mark.parametrize("shape", [synth.WORKLOADS["tiny"].model, MICRO_GQA],
                         ids=["fp32", "bf16"])
def test_eos_never_decoded_matches_plain_path(shape):
    """An <eos> id the generation never produces: the tracked path (host
    mirror, per-sequence geometry, per-step read-back) gives bit-identical
    logits and tokens to the plain path."""
    W = synth.Weights(shape, seed=2)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [26, 37])
    win = synth.WindowSettings(5, 6, 3, 2)
    s0, f0 = run_gpu(m, prompts, 22, win)
    used = set(np.concatenate(f0[0]).tolist())
    eos = next(v for v in range(shape.vocab - 1) if v not in used)
    ends = []
    s1, f1 = run_gpu(m, prompts, 22, win, eos_id=eos, ends=ends)
    m.free()
    assert ends == [len(p) + 22 for p in prompts]
    assert len(s0) == len(s1)
    for a, b in zip(s0, s1):
        assert a.logits.tobytes() == b.logits.tobytes()
        assert (a.positions == b.positions).all()
        assert (a.res.positions == b.res.positions).all()
    for b in range(2):
        np.testing.assert_array_equal(f0[0][b], f1[0][b])


def test_eos_argument_and_state_errors():
    shape = synth.WORKLOADS["tiny"].model
    W = synth.Weights(shape)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [10])
    for bad in (shape.mask_id, shape.vocab, -1):
        wc = wd.window_config(4, 4, 2, 1, eos_id=bad)
        with pytest.raises(wd.WdError) as e:
            wd.wd_prefill_prompt(m, prompts, 8, wc)
        assert e.value.status == wd.WD_ERR_INVALID_ARG
    wc = wd.window_config(4, 4, 2, 1)
    wc.stop_at_eos = 2
    with pytest.raises(wd.WdError) as e:
        wd.wd_prefill_prompt(m, prompts, 8, wc)
    assert e.value.status == wd.WD_ERR_INVALID_ARG
    gen = wd.wd_prefill_prompt(m, prompts, 8, wd.window_config(4, 4, 2, 1, eos_id=3))
    for fn in (wd.wd_slide_window, wd.wd_refresh_buffer):
        with pytest.raises(wd.WdError) as e:
            fn(gen)
        assert e.value.status == wd.WD_ERR_UNSUPPORTED
    assert list(wd.wd_seq_ends(gen)) == [18]
    gen.free()
    m.free()
