"""GPU parity: the HIP path through the C ABI against the CPU oracle, step by
step, on seeded inputs (see wdtest for the tolerances and the adoption
rules).  Runs on an MI355X only."""
import numpy as np
import pytest

import synth
from oracle.model import OracleModel
from oracle import generate_windowed
from wdtest import check_sequence, gpu_model, log, run_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)
import paper_2601_20332_amd as wd  # noqa: E402

# bf16 micro models: several GEMM tiles, ragged row tails, GQA and bias
MICRO_MHA = synth.ModelShape(n_layers=2, hidden=256, n_heads=2, n_kv_heads=2, head_dim=128,
                             ffn=512, vocab=1024, dtype=synth.DTYPE_BF16, rms_eps=1e-5,
                             rope_theta=10000.0)
MICRO_GQA = synth.ModelShape(n_layers=3, hidden=512, n_heads=4, n_kv_heads=2, head_dim=128,
                             ffn=1024, vocab=2048, dtype=synth.DTYPE_BF16, qkv_bias=True,
                             rms_eps=1e-6, rope_theta=1e6)


def _run_and_check(shape, prompts, G, win, full=False, seed=0, max_steps=None):
    log(f"[case] {shape} prompts={[len(p) for p in prompts]} G={G} win={win} full={full}")
    W = synth.Weights(shape, seed=seed)
    m = gpu_model(W)
    steps, final = run_gpu(m, prompts, G, win, full=full, max_steps=max_steps)
    log(f"[gpu] {len(steps)} steps")
    om = OracleModel(W)
    reps = []
    for b, p in enumerate(prompts):
        rep = check_sequence(om, p, G, win, steps, b, len(prompts), full=full,
                             max_steps=max_steps)
        log(f"[oracle] seq {b}: {rep}")
        print(f"PARITY {shape.dtype} L={shape.n_layers} H={shape.hidden} seq={b} steps={rep.steps} "
              f"max_rel_logit_err={rep.max_rel:.3e} adopted_sel={rep.select_adopted} "
              f"adopted_tok={rep.token_adopted}", flush=True)
        assert rep.steps == len(steps)
        if shape.dtype == synth.DTYPE_F32:
            assert rep.token_adopted == 0 and rep.select_adopted == 0
        reps.append(rep)
    m.free()
    return steps, final, reps


def test_tiny_fp32_whole_generation():
    w = synth.WORKLOADS["tiny"]
    prompts = synth.prompts(w.model, [w.prompt_len])
    steps, final, reps = _run_and_check(w.model, prompts, w.gen_len, w.window)
    assert len(steps) == 32
    # fp32: no adoption at all, final tokens identical to the oracle's own run
    assert reps[0].token_adopted == 0 and reps[0].select_adopted == 0
    x, _ = generate_windowed(OracleModel(synth.Weights(w.model)), prompts[0], w.gen_len, w.window)
    np.testing.assert_array_equal(final[0][0], x)
    assert final[1][0].all() and final[2] == 32


def test_tiny_fp32_full_sequence_path():
    w = synth.WORKLOADS["tiny"]
    prompts = synth.prompts(w.model, [w.prompt_len])
    steps, _, reps = _run_and_check(w.model, prompts, w.gen_len, w.window, full=True)
    assert reps[0].token_adopted == 0 and reps[0].select_adopted == 0


def test_tiny_fp32_batched_ragged():
    w = synth.WORKLOADS["tiny"]
    prompts = synth.prompts(w.model, [5, 32, 19])
    _run_and_check(w.model, prompts, 24, synth.WindowSettings(4, 6, 3, 2))


def test_bf16_mha_whole_generation():
    prompts = synth.prompts(MICRO_MHA, [70])
    _run_and_check(MICRO_MHA, prompts, 40, synth.WindowSettings(8, 16, 4, 1))


def test_bf16_gqa_bias_batched():
    prompts = synth.prompts(MICRO_GQA, [17, 81, 40])
    _run_and_check(MICRO_GQA, prompts, 30, synth.WindowSettings(6, 10, 3, 2))


# widths that are not multiples of 256 (hidden 384: Q/K/V 1152, O and down 384)
# take the 128-row-tile fallback above 64 rows; gate/up (1280) the LDS-pipelined
# tiles; rows 65-170 cover one and two row tiles and short K splits
MICRO_ODD = synth.ModelShape(n_layers=2, hidden=384, n_heads=3, n_kv_heads=3, head_dim=128,
                             ffn=640, vocab=1536, dtype=synth.DTYPE_BF16, rms_eps=1e-5,
                             rope_theta=10000.0)


# widths that are multiples of both 256 and 192 (Q/K/V 2304, gate/up 3072, O
# and down 768): the planner takes 192-feature tiles with K splits for all
# four above 96 rows; 90 + 170 prompt rows give ragged 128-row tiles
MICRO_W768 = synth.ModelShape(n_layers=2, hidden=768, n_heads=6, n_kv_heads=6, head_dim=128,
                              ffn=1536, vocab=2048, dtype=synth.DTYPE_BF16, rms_eps=1e-5,
                              rope_theta=10000.0)


def test_bf16_many_row_kernels_192_feature_tiles():
    prompts = synth.prompts(MICRO_W768, [90, 170])
    _run_and_check(MICRO_W768, prompts, 48, synth.WindowSettings(8, 32, 4, 2))


def test_bf16_many_row_kernels_odd_widths():
    prompts = synth.prompts(MICRO_ODD, [65, 100])
    _run_and_check(MICRO_ODD, prompts, 40, synth.WindowSettings(8, 24, 4, 2))


def test_bf16_full_sequence_path():
    prompts = synth.prompts(MICRO_GQA, [20, 9])
    _run_and_check(MICRO_GQA, prompts, 12, synth.WindowSettings(4, 4, 2, 2), full=True)


def test_bf16_edge_windows():
    """Window wider than the generation, R = 1, early phase end (R*k > E),
    empty buffer, n_active > remaining."""
    prompts = synth.prompts(MICRO_MHA, [3])
    for win in [synth.WindowSettings(64, 64, 1, 3), synth.WindowSettings(2, 0, 5, 1),
                synth.WindowSettings(3, 1, 8, 2)]:
        _run_and_check(MICRO_MHA, prompts, 10, win)


def test_bf16_gqa_refresh_rows_grouped_attention():
    """Refresh steps of 300 and more rows with grouped K/V heads take the
    attention kernel whose workgroups serve all query heads of a K/V head
    (normal steps keep one workgroup per query head)."""
    prompts = synth.prompts(MICRO_GQA, [300, 260])
    steps, _, _ = _run_and_check(MICRO_GQA, prompts, 20, synth.WindowSettings(6, 10, 4, 2))
    assert steps[0].res.is_refresh and steps[0].res.n_rows >= 2 * 256


def test_bf16_pruning_only_every_step_refreshes():
    """Window pruning without the cache (the Table 1 setting of Sec. 5.2): R =
    1, so every step is a refresh over the retained prefix [0, c), with E = 8
    well below G = 24 (far-field positions pruned at every step)."""
    prompts = synth.prompts(MICRO_GQA, [17, 40])
    steps, _, _ = _run_and_check(MICRO_GQA, prompts, 24, synth.WindowSettings(4, 4, 1, 1))
    assert all(s.res.is_refresh for s in steps)
    # rows = c = the E-th undecoded position + 1, per sequence: below S until
    # fewer than E undecoded positions remain
    assert steps[0].res.n_rows == (17 + 8) + (40 + 8)


@pytest.mark.parametrize("dtype_shape", [synth.WORKLOADS["tiny"].model, MICRO_GQA])
def test_refresh_cache_equals_oracle_kv(dtype_shape):
    """After a refresh step the cache holds K/V of the forward over [0, c)."""
    shape = dtype_shape
    log(f"[case] kv after refresh {shape}")
    W = synth.Weights(shape, seed=3)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [37, 12])
    G = 20
    win = synth.WindowSettings(4, 6, 4, 1)
    gen = wd.wd_prefill_prompt(m, prompts, G, wd.window_config(4, 6, 4, 1))
    wd.wd_step(gen)
    om = OracleModel(W)
    for b, p in enumerate(prompts):
        x = np.concatenate([p, np.full(G, shape.mask_id)])
        c = len(p) + win.external
        _, K, V = om.forward(x[:c])
        for l in range(shape.n_layers):
            k, v = wd.wd_debug_kv(gen, l, b)
            assert k.shape[0] == c
            for got, ref in ((k, K[l]), (v, V[l])):
                err = np.abs(got - ref).max() / np.abs(ref).max()
                assert err <= (1e-5 if shape.dtype == synth.DTYPE_F32 else 2e-2), err
                if shape.dtype == synth.DTYPE_BF16 and l == 0:
                    # first layer: both sides round the same values to bf16, so
                    # nearly every element is identical (deeper layers inherit
                    # rounding flips, which this random-init model amplifies)
                    assert np.mean(got == ref) > 0.999
    gen.free()
    m.free()


def test_step_after_completion_is_a_state_error():
    shape = MICRO_MHA
    m = gpu_model(synth.Weights(shape))
    gen = wd.wd_prefill_prompt(m, synth.prompts(shape, [4]), 3, wd.window_config(2, 2, 2, 2))
    while True:
        try:
            wd.wd_step(gen)
        except wd.WdError as e:
            assert e.status == wd.WD_ERR_STATE
            break
    with pytest.raises(wd.WdError) as ei:
        wd.wd_full_step(gen)
    assert ei.value.status == wd.WD_ERR_STATE
    with pytest.raises(wd.WdError):
        wd.wd_refresh_buffer(gen)
    gen.free()
    m.free()


def test_explicit_slide_and_refresh_match_automatic_steps():
    shape = MICRO_MHA
    W = synth.Weights(shape, seed=5)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [30])
    wc = wd.window_config(4, 8, 3, 1)
    a = wd.wd_prefill_prompt(m, prompts, 16, wc)
    b = wd.wd_prefill_prompt(m, prompts, 16, wc)
    wd.wd_slide_window(b)
    wd.wd_refresh_buffer(b)
    with pytest.raises(wd.WdError):
        wd.wd_refresh_buffer(b)
    for _ in range(16):
        ra, rb = wd.wd_step(a), wd.wd_step(b)
        assert ra.positions.tolist() == rb.positions.tolist()
        assert ra.tokens.tolist() == rb.tokens.tolist()
        assert ra.conf.tobytes() == rb.conf.tobytes()
    a.free()
    b.free()
    m.free()


def test_deterministic_runs():
    shape = MICRO_GQA
    W = synth.Weights(shape, seed=9)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [33, 50])
    win = synth.WindowSettings(5, 7, 4, 2)
    s1, f1 = run_gpu(m, prompts, 20, win)
    s2, f2 = run_gpu(m, prompts, 20, win)
    for x, y in zip(s1, s2):
        assert x.logits.tobytes() == y.logits.tobytes()
    for b in range(2):
        np.testing.assert_array_equal(f1[0][b], f2[0][b])
    m.free()


def test_profile_records_by_kernel_class():
    """Timing records: every GEMM launch lands in exactly one kernel class, the
    many-row refresh products in the 128-row-tile kernel and the few-row normal
    steps in the weight-streaming kernel; algorithmic bytes follow the stated
    formula; an unknown class is rejected."""
    shape = MICRO_GQA
    W = synth.Weights(shape, seed=4)
    m = gpu_model(W)
    prompts = synth.prompts(shape, [60, 70])          # refresh rows > 64, normal rows <= 64
    win = synth.WindowSettings(6, 10, 4, 2)
    wd.wd_profile_enable(m, True)
    run_gpu(m, prompts, 16, win, max_steps=4, keep_logits=False)   # steps 0-3: one refresh
    n_all, ms_all, by_all, fl_all = wd.wd_profile_read(m, wd.WD_PROF_ALL)
    n_rows, ms_rows, by_rows, _ = wd.wd_profile_read(m, wd.WD_PROF_GEMM_ROWS)
    n_tiled, ms_tiled, by_tiled, _ = wd.wd_profile_read(m, wd.WD_PROF_GEMM_TILED)
    n_f32 = wd.wd_profile_read(m, wd.WD_PROF_GEMM_F32)[0]
    n_attn, ms_attn, by_attn, fl_attn = wd.wd_profile_read(m, wd.WD_PROF_ATTN)
    assert n_rows > 0 and n_tiled > 0 and n_f32 == 0
    assert n_all == n_rows + n_tiled + n_attn
    assert ms_all > 0 and abs(ms_all - ms_rows - ms_tiled - ms_attn) <= 1e-6 * ms_all
    assert abs(by_all - by_rows - by_tiled - by_attn) <= 1e-9 * by_all
    # one refresh step: 4 projections per layer through the tiled kernel
    assert n_tiled == 4 * shape.n_layers
    # attention: one unit per layer and step; K/V of [0, c) plus q and output rows
    assert n_attn == 4 * shape.n_layers and ms_attn > 0
    wc = wd.window_config(win.n_active, win.n_buffer, win.refresh_every, win.unmask_per_step)
    want_by = want_fl = 0.0
    for p in prompts:
        plan = wd.wd_plan(len(p), 16, wc)
        for t in range(4):
            c, r = int(plan["ctx_len"][t]), int(plan["n_rows"][t])
            want_by += 2.0 * c * shape.n_kv_heads * shape.head_dim * 2
            want_by += 2.0 * r * shape.n_heads * shape.head_dim * 2
            want_fl += 4.0 * r * c * shape.n_heads * shape.head_dim
    assert by_attn == pytest.approx(want_by * shape.n_layers, rel=1e-12)
    assert fl_attn == pytest.approx(want_fl * shape.n_layers, rel=1e-12)
    # reading does not consume the records; enabling again discards them
    assert wd.wd_profile_read(m, wd.WD_PROF_ALL)[0] == n_all
    wd.wd_profile_enable(m, True)
    assert wd.wd_profile_read(m, wd.WD_PROF_ALL)[0] == 0
    with pytest.raises(wd.WdError):
        wd.wd_profile_read(m, 7)
    wd.wd_profile_enable(m, False)
    m.free()


def test_measured_peaks_are_plausible():
    """The peak probe's two kernels run and report numbers of the right order
    for an MI355X (vendor peaks: 2.5 PFLOP/s dense bf16, 8 TB/s)."""
    W = synth.Weights(MICRO_MHA)
    m = gpu_model(W)
    try:
        tflops, gbs = wd.wd_measure_peaks(m)
    finally:
        m.free()
    print(f"PEAKS mfma_bf16={tflops:.1f} TFLOP/s hbm_read={gbs:.1f} GB/s", flush=True)
    assert 200.0 < tflops < 2600.0
    assert 1000.0 < gbs < 8200.0
