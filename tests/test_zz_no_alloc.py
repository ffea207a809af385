"""wd_step_noalloc, the step whose scratch lives in the library's static
device array: through the C ABI, two generations in a row (the second with a
smaller input) must equal wd_step's bit for bit, every step (positions,
tokens, confidences, active-row logits) and in the final state.  A step
whose scratch would not fit is refused before it changes anything, and the
settings the entry point does not take are refused.  Runs on an MI355X
only."""
import numpy as np
import pytest

import synth
from wdtest import gpu_model, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)
import paper_2601_20332_amd as wd  # noqa: E402

# widths that take the many-row kernels with K splits on refresh steps (so the
# split-K partials are used), split-KV attention on normal steps and, with
# 192 vocabulary tiles, the LM head with the confidence reduction inside
SHAPE = synth.ModelShape(n_layers=2, hidden=768, n_heads=6, n_kv_heads=6, head_dim=128,
                         ffn=1536, vocab=192 * 64, dtype=synth.DTYPE_BF16, rms_eps=1e-5,
                         rope_theta=10000.0)


def _drive(model, prompts, G, win, step):
    wc = wd.window_config(*win)
    gen = wd.wd_prefill_prompt(model, prompts, G, wc)
    out = []
    try:
        wd.wd_debug_keep_logits(gen, True)
        while True:
            try:
                r = step(gen)
            except wd.WdError as e:
                if e.status == wd.WD_ERR_STATE:
                    break
                raise
            lg, pos = wd.wd_debug_logits(gen)
            out.append((r, lg, pos))
        final = wd.wd_get_state(gen)
    finally:
        gen.free()
    return out, final


def _same(a, b):
    (sa, fa), (sb, fb) = a, b
    assert len(sa) == len(sb) > 0
    for t, ((ra, la, pa), (rb, lb, pb)) in enumerate(zip(sa, sb)):
        assert (ra.step, ra.is_refresh, ra.n_rows, ra.n_selected) == \
            (rb.step, rb.is_refresh, rb.n_rows, rb.n_selected), t
        assert ra.positions.tobytes() == rb.positions.tobytes(), t
        assert ra.tokens.tobytes() == rb.tokens.tobytes(), t
        assert ra.conf.tobytes() == rb.conf.tobytes(), t
        assert pa.tobytes() == pb.tobytes() and la.tobytes() == lb.tobytes(), t
    for x, y in zip(fa[0], fb[0]):
        np.testing.assert_array_equal(x, y)
    assert fa[2] == fb[2]
    return len(sa)


def test_noalloc_steps_equal_wd_step_twice_second_smaller():
    m = gpu_model(synth.Weights(SHAPE, seed=17))
    try:
        cases = [([90, 170], 48, (8, 32, 4, 2)),    # refresh steps of 338 and more rows
                 ([12], 16, (4, 4, 3, 1))]           # then a smaller input
        for lens, G, win in cases:
            log(f"[case] wd_step_noalloc vs wd_step, prompts {lens}, G {G}, window {win}")
            prompts = synth.prompts(SHAPE, lens)
            ref = _drive(m, prompts, G, win, wd.wd_step)
            got = _drive(m, prompts, G, win, wd.wd_step_noalloc)
            n = _same(got, ref)
            print(f"NOALLOC prompts={lens} G={G} steps={n} identical to wd_step", flush=True)
    finally:
        m.free()


# one 4096-wide layer: the output projection writes split-K partials of at
# least rows x 4096 x 4 bytes, whatever its split count
WIDE = synth.ModelShape(n_layers=1, hidden=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                        ffn=4096, vocab=192 * 64, dtype=synth.DTYPE_BF16, rms_eps=1e-5,
                        rope_theta=10000.0)


def test_noalloc_refuses_what_does_not_fit_and_leaves_the_sequence_untouched():
    m = gpu_model(synth.Weights(WIDE, seed=5))
    try:
        # the first refresh runs 4 x (2000 + 40) rows: its O partials alone
        # (8160 x 4096 x 4 bytes) exceed the 96 MiB static scratch
        prompts = synth.prompts(WIDE, [2000] * 4)
        gen = wd.wd_prefill_prompt(m, prompts, 24, wd.window_config(8, 32, 4, 2))
        with pytest.raises(wd.WdError) as ei:
            wd.wd_step_noalloc(gen)
        assert ei.value.status == wd.WD_ERR_OUT_OF_MEMORY
        assert "static scratch" in str(ei.value)
        r = wd.wd_step(gen)                # the step the refusal left untaken
        assert r.step == 0 and r.is_refresh
        wd.wd_get_state(gen)
        gen.free()
    finally:
        m.free()
    m = gpu_model(synth.Weights(SHAPE, seed=17))
    try:
        # settings it does not take
        eos = wd.wd_prefill_prompt(m, synth.prompts(SHAPE, [20]), 8,
                                   wd.window_config(4, 4, 2, 1, eos_id=5))
        with pytest.raises(wd.WdError) as ei:
            wd.wd_step_noalloc(eos)
        assert ei.value.status == wd.WD_ERR_UNSUPPORTED
        eos.free()
        gen = wd.wd_prefill_prompt(m, synth.prompts(SHAPE, [20]), 8, wd.window_config(4, 4, 2, 1))
        wd.wd_profile_enable(m, True)
        with pytest.raises(wd.WdError) as ei:
            wd.wd_step_noalloc(gen)
        assert ei.value.status == wd.WD_ERR_UNSUPPORTED
        wd.wd_profile_enable(m, False)
        assert wd.wd_step_noalloc(gen).step == 0
        gen.free()
    finally:
        m.free()
