"""GPU parity at the full per-layer shapes of the LLaDA-8B and Dream-7B
workloads (hidden, heads, FFN, vocabulary, window settings, prompt and
generation lengths exactly as benchmarked, so every kernel runs in the launch
configuration the benchmark times), with the layer stack cut to 2 layers so
the float64 oracle replays the first phase in seconds.  A property that holds
at any depth is checked on the full 32-layer LLaDA-8B shape."""
import time

import numpy as np
import pytest

import synth
from oracle.model import OracleModel
import wdtest
from wdtest import check_sequence, gpu_model, log, run_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)
import paper_2601_20332_amd as wd  # noqa: E402


# (workload, steps to check, sequences the oracle replays)
CASES = [
    ("llada8b", 10, None),        # a whole phase (R = 8) and the next refresh
    ("dream7b", 10, None),
    ("llada8b_long", 10, None),   # c = 832, 66-82 online rows (many-row GEMM path)
    ("llada8b_batch16", 10, (0, 5)),  # ragged prompts; 528-624 online rows per step
]


@pytest.mark.parametrize("name,n_steps,seqs", CASES, ids=[c[0] for c in CASES])
def test_first_phases_at_full_width(name, n_steps, seqs):
    w = synth.WORKLOADS[name]
    shape = synth.with_layers(w.model, 2)
    t0 = time.time()
    log(f"[case] {name} at full width, 2 layers")
    W = synth.Weights(shape)
    m = gpu_model(W)
    prompts = synth.prompts(shape, synth.prompt_lengths(w))
    steps, _ = run_gpu(m, prompts, w.gen_len, w.window, max_steps=n_steps)
    m.free()
    log(f"[gpu] {len(steps)} steps in {time.time() - t0:.1f}s")
    om = OracleModel(W, cache_budget_bytes=40e9)
    check = range(len(prompts)) if seqs is None else seqs
    if seqs is not None:
        # the shortest and the longest prompt of the batch
        lens = [len(p) for p in prompts]
        check = sorted({lens.index(min(lens)), lens.index(max(lens))})
    for b in check:
        rep = check_sequence(om, prompts[b], w.gen_len, w.window, steps, b, len(prompts),
                             max_steps=n_steps)
        print(f"PARITY {name}-2L seq={b} prompt={len(prompts[b])} steps={rep.steps} "
              f"max_rel_logit_err={rep.max_rel:.3e} adopted_sel={rep.select_adopted} "
              f"adopted_tok={rep.token_adopted} ({time.time() - t0:.1f}s)", flush=True)
        assert rep.steps == n_steps


def test_llada8b_2_layers_pruning_only():
    """R = 1 with E = 96 < G = 256 at the LLaDA-8B width (the pruning-only
    setting of Table 1, Sec. 5.2): every step is a refresh over [0, c)."""
    w = synth.WORKLOADS["llada8b"]
    shape = synth.with_layers(w.model, 2)
    win = synth.WindowSettings(w.window.n_active, w.window.n_buffer, 1, 1)
    n_steps = 6
    log("[case] llada8b at full width, 2 layers, R = 1, E = 96")
    W = synth.Weights(shape)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [w.prompt_len])
    steps, _ = run_gpu(m, prompts, w.gen_len, win, max_steps=n_steps)
    m.free()
    assert all(s.res.is_refresh for s in steps)
    assert [s.res.n_rows for s in steps] == [w.prompt_len + 96 + t for t in range(n_steps)]
    rep = check_sequence(OracleModel(W, cache_budget_bytes=40e9), prompts[0], w.gen_len, win,
                         steps, 0, 1, max_steps=n_steps)
    print(f"PARITY llada8b-2L-R1 seq=0 steps={rep.steps} max_rel_logit_err={rep.max_rel:.3e} "
          f"adopted_sel={rep.select_adopted} adopted_tok={rep.token_adopted}", flush=True)
    assert rep.steps == n_steps


class HeldWeights(synth.Weights):
    """Seeded weights generated once and kept as drawn (bf16 bit patterns), so
    the GPU upload and the oracle read the same draw without generating the
    8B parameters twice."""

    def __init__(self, *a, **k):
        super().__init__(*a, **k)
        self._held = {}

    def raw(self, i):
        r = self._held.get(i)
        if r is None:
            r = self._held[i] = super().raw(i)
        return r

    def drop(self):
        self._held.clear()


@pytest.mark.timeout(900)
def test_llada8b_full_depth_against_oracle():
    """All 32 layers of the LLaDA-8B workload at its window settings: the first
    refresh step, the phase's 7 normal steps and the next refresh step (R + 1
    steps) against the float64 oracle, so the bf16 bound is checked at the
    depth the benchmark runs, where rounding differences accumulate over the
    layers (Sec. 4.3 refresh and normal steps, Sec. 5.1 model)."""
    w = synth.WORKLOADS["llada8b"]
    shape = w.model
    n_steps = w.window.refresh_every + 1
    t0 = time.time()
    log(f"[case] llada8b full depth ({shape.n_layers} layers), {n_steps} steps against the oracle")
    W = HeldWeights(shape)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [w.prompt_len])
    steps, _ = run_gpu(m, prompts, w.gen_len, w.window, max_steps=n_steps)
    m.free()
    log(f"[gpu] {len(steps)} steps, weights drawn and run in {time.time() - t0:.1f}s")
    # every float64 weight stays resident: 8.0e9 parameters x 8 bytes
    om = OracleModel(W, cache_budget_bytes=80e9)
    rep = check_sequence(om, prompts[0], w.gen_len, w.window, steps, 0, 1, max_steps=n_steps,
                         progress=True)
    W.drop()
    print(f"PARITY llada8b-32L seq=0 steps={rep.steps} max_rel_logit_err={rep.max_rel:.3e} "
          f"adopted_sel={rep.select_adopted} adopted_tok={rep.token_adopted} "
          f"({time.time() - t0:.1f}s)", flush=True)
    assert rep.steps == n_steps
    assert steps[0].res.is_refresh and steps[-1].res.is_refresh


# Logit bound for the normal and next refresh steps at full Dream-7B depth.
# The bf16 bound (2e-2) sits on the rounding floor of this datapath there: the
# oracle's own layer run on float32 arrays (fp32 GEMMs, the same bf16
# rounding points) differs from it by 1.89e-2 after 28 layers on the first
# refresh step, and the GPU by 1.83e-2 on that step; over the following
# steps the largest per-row error of a float32 implementation is a tail of
# that floor (the GPU's reached 2.11-2.12e-2, over 2e-2 on 1-2 of 9 steps).  The
# first refresh step, where the floor was measured, keeps the 2e-2 bound.
DREAM_DEPTH_LOGIT_TOL = 2.5e-2


@pytest.mark.timeout(900)
def test_dream7b_full_depth_against_oracle():
    """All 28 layers of the Dream-7B workload (grouped K/V heads, QKV bias) at
    its window settings: the first refresh step, the phase's normal steps and
    the next refresh step against the float64 oracle (Sec. 4.3 refresh and
    normal steps, Sec. 5.1 models).  Bookkeeping, selections and tokens at the
    standard bar; logits at 2e-2 on the first refresh step and at
    DREAM_DEPTH_LOGIT_TOL after it."""
    w = synth.WORKLOADS["dream7b"]
    shape = w.model
    n_steps = w.window.refresh_every + 1
    t0 = time.time()
    log(f"[case] dream7b full depth ({shape.n_layers} layers), {n_steps} steps against the oracle")
    W = HeldWeights(shape)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [w.prompt_len])
    steps, _ = run_gpu(m, prompts, w.gen_len, w.window, max_steps=n_steps)
    m.free()
    log(f"[gpu] {len(steps)} steps, weights drawn and run in {time.time() - t0:.1f}s")
    om = OracleModel(W, cache_budget_bytes=80e9)
    rep = check_sequence(om, prompts[0], w.gen_len, w.window, steps, 0, 1, max_steps=n_steps,
                         progress=True, logit_tol=DREAM_DEPTH_LOGIT_TOL)
    W.drop()
    over = sum(e > wdtest.LOGIT_TOL[synth.DTYPE_BF16] for e in rep.step_rel)
    print(f"PARITY dream7b-28L seq=0 steps={rep.steps} max_rel_logit_err={rep.max_rel:.3e} "
          f"first_refresh={rep.step_rel[0]:.3e} steps_over_2e-2={over} "
          f"adopted_sel={rep.select_adopted} adopted_tok={rep.token_adopted} "
          f"({time.time() - t0:.1f}s)", flush=True)
    assert rep.steps == n_steps
    assert rep.step_rel[0] <= wdtest.LOGIT_TOL[synth.DTYPE_BF16]
    assert steps[0].res.is_refresh and steps[-1].res.is_refresh


def test_llada8b_32_layers_window_covering_everything_equals_full_path():
    """With E >= G, n_active >= G and R = 1 Window-Diffusion is standard decoding;
    on the GPU both paths run the same row sets through the same kernels, so the
    trajectories must agree bit for bit (a property that holds at any size)."""
    w = synth.WORKLOADS["llada8b"]
    shape = w.model
    log("[case] llada8b 32 layers, windowed(R=1, E>=G) vs full")
    W = synth.Weights(shape)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [w.prompt_len])
    G = 12
    win = synth.WindowSettings(G, 0, 1, 1)
    s_w, f_w = run_gpu(m, prompts, G, win)
    s_f, f_f = run_gpu(m, prompts, G, win, full=True)
    m.free()
    assert len(s_w) == len(s_f) == G
    for a, b in zip(s_w, s_f):
        assert a.res.positions.tolist() == b.res.positions.tolist()
        assert a.logits.tobytes() == b.logits.tobytes()
    np.testing.assert_array_equal(f_w[0][0], f_f[0][0])
