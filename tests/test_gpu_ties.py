"""The update rule's tie break (Sec. 3.1 update set: the k most confident
candidates; equal confidences go to the lowest position) under exact ties.

An all-zero LM head gives every active row the same logits (all zero), so
every candidate has the same confidence, 1 / (vocab - 1), in any precision,
and the same prediction, the lowest non-[MASK] id (0).  Each step must then
decode the lowest positions of the active set, in increasing order, with
token 0, bit-exact against the oracle and with no adoption.  Covered: the
fused LM head (bf16, at most 64 active rows), the unfused bf16 LM head with
its two-pass confidence (more rows), the fp32 path and the full-sequence
step.  Runs on an MI355X only."""
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

# 192 vocabulary tiles of 64: the smallest vocabulary the fused LM head takes
BF16_SHAPE = synth.ModelShape(n_layers=2, hidden=256, n_heads=2, n_kv_heads=2, head_dim=128,
                              ffn=512, vocab=192 * 64, dtype=synth.DTYPE_BF16)


class ZeroHead(synth.Weights):
    def raw(self, i):
        r = super().raw(i)
        return np.zeros_like(r) if self.specs[i][0] == "lm_head" else r


def _check_ties(shape, prompt_lens, G, win, full=False, expect_rows=None):
    log(f"[case] exact ties {shape.dtype} vocab {shape.vocab} prompts={prompt_lens} win={win} "
        f"full={full}")
    W = ZeroHead(shape, seed=13)
    m = gpu_model(W)
    prompts = synth.prompts(shape, prompt_lens)
    steps, final = run_gpu(m, prompts, G, win, full=full)
    m.free()
    B = len(prompts)
    if expect_rows is not None:
        assert len(steps[0].positions) == expect_rows
    k = win.unmask_per_step
    for t, gs in enumerate(steps):
        n = len(gs.positions) // B
        assert not gs.logits.any(), f"step {t}: non-zero logits from a zero LM head"
        for b in range(B):
            act = [int(p) for p in gs.positions[b * n:(b + 1) * n] if p >= 0]
            assert act == sorted(act)
            want = act[:min(k, len(act))]
            got = [int(p) for p in gs.res.positions[b] if p >= 0]
            assert got == want, f"step {t} seq {b}: decoded {got}, lowest positions {want}"
            assert all(int(x) == 0 for x in gs.res.tokens[b][:len(got)])
            conf = gs.res.conf[b][:len(got)]
            assert (conf == conf[0]).all()
            assert abs(float(conf[0]) * (shape.vocab - 1) - 1.0) < 1e-6
    om = OracleModel(W)
    for b, p in enumerate(prompts):
        rep = check_sequence(om, p, G, win, steps, b, B, full=full, max_adopt_frac=0.0)
        assert rep.select_adopted == 0 and rep.token_adopted == 0
        assert rep.steps == len(steps)
        print(f"PARITY-TIES {shape.dtype} seq={b} steps={rep.steps} max_rel_logit_err={rep.max_rel:.1e} "
              f"adopted_sel=0 adopted_tok=0", flush=True)
    for b in range(B):
        gen = final[0][b][len(prompts[b]):]
        assert (gen == 0).all() and final[1][b].all()


def test_ties_fused_lm_head():
    # 2 sequences x 16 active rows: the LM head reduces its tiles itself
    _check_ties(BF16_SHAPE, [24, 40], 48, synth.WindowSettings(16, 16, 4, 2), expect_rows=32)


def test_ties_unfused_lm_head():
    # 3 sequences x 32 active rows = 96 rows: stored logits, two-pass confidence
    _check_ties(BF16_SHAPE, [24, 40, 31], 48, synth.WindowSettings(32, 16, 4, 3), expect_rows=96)


def test_ties_fp32():
    _check_ties(synth.WORKLOADS["tiny"].model, [10, 20], 24, synth.WindowSettings(8, 16, 4, 2))


def test_ties_full_sequence_step():
    _check_ties(BF16_SHAPE, [9, 30], 20, synth.WindowSettings(4, 4, 2, 2), full=True)
