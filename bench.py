#!/usr/bin/env python3
"""Throughput of Window-Diffusion decoding on one MI355X.

Workload (default): the LLaDA-8B shape in bf16 (32 layers, hidden 4096,
32 heads x 128, SwiGLU 12288, vocabulary 126464) with seeded random-init
weights N(0, 0.02); batch 1, a 128-token random prompt and 256 masked
positions; 32 active + 64 buffer positions, refresh every 8 steps, 1 token
unmasked per step.

One bench step is one whole generation: wd_prefill_prompt plus every
denoising step (refresh and normal steps) until all 256 positions are
decoded.  `value` is denoising steps per second over the timed generations.
Also reported: decoded tokens/s, the speedup over standard full-sequence
decoding on the same GPU and kernels, the roofline of the dominant kernel
(the few-row projection GEMM of the normal steps, k_gemm_bf16, timed with HIP
events on the library's stream; HBM bound), the same for the many-row GEMM
of the refresh steps (k_gemm_bf16_dma; MFMA bound), adaptive termination at
<eos> on the same workload (an <eos> id taken from the fixed-length run), the
buffer-only refresh variant (not the paper's method), the FP8-weight variant
(not the paper's precision), the same model on the long generation (512 +
1024, with its full-sequence comparison) and on the ragged batch of 16, the
Dream-7B shape, and the CPU oracle on a bounded sample of the same workload.
Every generation ends with a read of the device's own checks of its steps;
a failed check raises, so no record is printed for it.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "denoising steps/s + decoded tokens/s at LLaDA-8B shape, 1 GPU; MFMA/HBM % peak"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "kernel_traffic.json")
CSRC = os.path.join(ROOT, "paper_2601_20332_amd", "csrc")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# kernel classes of wd_profile_read, the kernel each one is named by, and the
# source file that holds it (its hash gates the stored counter traffic)
KERNEL_CLASSES = {1: "k_gemm_bf16", 2: "k_gemm_bf16_dma", 4: "k_attn_bf16"}
PROFILE_NAMES = KERNEL_CLASSES
KERNEL_SOURCES = {"k_gemm_bf16": "gemm.hip", "k_gemm_bf16_dma": "gemm_tiles.hip",
                  "k_attn_bf16": "layer.hip"}


def source_hash(kernel: str) -> str:
    path = os.path.join(CSRC, KERNEL_SOURCES[kernel])
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def measured_traffic(kernel: str):
    """HBM bytes per launch (per unit for attention) of one kernel class from the
    committed rocprofv3 counter runs, if they were taken on the current source
    of that kernel."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    k = rec.get("kernels", {}).get(kernel, {})
    if not k or k.get("source_sha256_16") != source_hash(kernel):
        return None
    return k.get("hbm_bytes_per_launch")


def kernel_class_of(name: str):
    """WD_PROF_* class of a kernel name as rocprofv3 prints it: the few-row
    products (k_gemm_bf16, and k_gemm_bf16_fused that carries the Q/K/V or
    SwiGLU epilogue), the many-row kernels (k_gemm_bf16_dma; k_gemm_bf16_big
    where the former does not apply: fp8 weights, widths not a multiple of
    256), or one layer's bf16 attention (k_attn_bf16 and its split merge
    k_attn_combine)."""
    if "k_gemm_bf16_dma<" in name or "k_gemm_bf16_big<" in name:
        return 2
    if "k_gemm_bf16<" in name or "k_gemm_bf16_fused<" in name:
        return 1
    if "k_attn_bf16" in name or "k_attn_combine" in name:
        return 4
    return None


def starts_unit(name: str) -> bool:
    """Whether a dispatch starts a timing unit: every GEMM launch does; an
    attention unit is k_attn_bf16 plus the k_attn_combine that may follow it."""
    return "k_attn_combine" not in name


def read_counter_csv(folder: str):
    """(kernel name, counter value) rows of a rocprofv3 --pmc -f csv output folder."""
    import csv
    import glob
    files = glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        sys.exit(f"no counter_collection.csv under {folder}")
    rows = []
    for f in files:
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                rows.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return rows


def pmc_summary(gemm_fetch: str, gemm_write: str, copy_fetch: str, copy_write: str,
                copy_mib: int):
    """Turn the four rocprofv3 counter runs (FETCH_SIZE and WRITE_SIZE, in KiB per
    dispatch, over one generation and over plain copies of copy_mib MiB) into HBM
    bytes per launch of each GEMM kernel and per layer of attention; writes
    TRAFFIC_FILE and prints a table."""
    copy_bytes = copy_mib << 20

    def copy_scale(folder):
        vals = [v for n, v in read_counter_csv(folder) if "copyBuffer" in n]
        if not vals:
            sys.exit(f"no copy dispatch in {folder}")
        return copy_bytes / (sum(vals) / len(vals))

    sf, sw = copy_scale(copy_fetch), copy_scale(copy_write)
    per = {}
    for folder, key, scale in ((gemm_fetch, "fetch", sf), (gemm_write, "write", sw)):
        for name, v in read_counter_csv(folder):
            cls = kernel_class_of(name)
            if cls is None:
                continue
            k = KERNEL_CLASSES[cls]
            d = per.setdefault(k, {"fetch": [], "write": [], "fetch_units": 0, "write_units": 0,
                                   "instances": {}})
            d[key].append(v * scale)
            d[key + "_units"] += starts_unit(name)
            inst = name.split("(")[0].replace("void ", "")
            di = d["instances"].setdefault(inst, {"fetch": [], "write": []})
            di[key].append(v * scale)
    kernels = {}
    lines = ["| kernel instance | dispatches | fetched MB / dispatch | written MB / dispatch |",
             "|---|---|---|---|"]
    for k, d in per.items():
        if len(d["fetch"]) != len(d["write"]) or d["fetch_units"] != d["write_units"]:
            sys.exit(f"{k}: {len(d['fetch'])} FETCH_SIZE vs {len(d['write'])} WRITE_SIZE dispatches")
        n = d["fetch_units"]
        f, w = sum(d["fetch"]) / n, sum(d["write"]) / n
        kernels[k] = {"source": KERNEL_SOURCES[k], "source_sha256_16": source_hash(k),
                      "dispatches": len(d["fetch"]), "units": n,
                      "hbm_fetch_bytes_per_launch": round(f),
                      "hbm_write_bytes_per_launch": round(w), "hbm_bytes_per_launch": round(f + w)}
        for inst, di in sorted(d["instances"].items(), key=lambda x: -len(x[1]["fetch"])):
            m = len(di["fetch"])
            lines.append(f"| `{inst}` | {m} | {sum(di['fetch']) / m / 1e6:.1f} | "
                         f"{sum(di['write']) / max(1, len(di['write'])) / 1e6:.2f} |")
    rec = {"copy_mib": copy_mib,
           "fetch_bytes_per_count": round(sf, 4), "write_bytes_per_count": round(sw, 4),
           "kernels": kernels}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec, indent=1))
    print("\n".join(lines))


def roofline_of(model, kernel_class: int, elapsed_ev: float):
    """Roofline entry of one GEMM kernel from the event-timed launches of the
    instrumented pass: the few-row kernel streams its weights (HBM bound), the
    many-row kernel is priced against dense bf16 MFMA."""
    import paper_2601_20332_amd as wd
    launches, ms, alg_bytes, alg_flops = wd.wd_profile_read(model, kernel_class)
    if launches <= 0 or ms <= 0:
        return None
    name = PROFILE_NAMES[kernel_class]
    avg_s = ms / 1e3 / launches
    gbs = alg_bytes / launches / avg_s / 1e9
    tfs = alg_flops / launches / avg_s / 1e12
    hbm = kernel_class in (1, 4)
    achieved, peak = (gbs, HBM_PEAK_GBS) if hbm else (tfs, BF16_PEAK_TFLOPS)
    label = {1: " + k_gemm_bf16_fused (at most 64 rows; 96 for gate/up, O, down)", 2: " (more rows)",
             4: " + k_attn_combine (one layer's attention)"}[kernel_class]
    return {
        "kernel": name + label,
        "bound": "hbm" if hbm else "mfma",
        "achieved": round(achieved, 1),
        "peak": peak,
        "unit": "GB/s" if hbm else "TFLOP/s",
        "frac": round(achieved / peak, 4),
        "traffic": measured_traffic(name),
        "launches": launches,
        "avg_launch_us": round(avg_s * 1e6, 2),
        "alg_bytes_per_launch": round(alg_bytes / launches),
        "alg_flops_per_launch": round(alg_flops / launches),
        "alg_gbs": round(gbs, 1),
        "tflops": round(tfs, 1),
        "share_of_step_time": round(ms / 1e3 / elapsed_ev, 3),
    }


def upload_model(shape, device, fp8_too=False):
    """Packs the seeded weights into the library (and, with fp8_too, a second
    model of the FP8-weight variant from the same device tensors)."""
    import numpy as np
    import torch
    import synth
    import paper_2601_20332_amd as wd
    W = synth.Weights(shape)
    ts = []
    for _, raw in W.iter_raw(workers=min(16, os.cpu_count() or 4)):
        a = raw.view(np.int16) if raw.dtype == np.uint16 else raw
        ts.append(torch.from_numpy(np.ascontiguousarray(a)).to(device))

    def cfg(fp8):
        return wd.model_config(n_layers=shape.n_layers, hidden=shape.hidden,
                               n_heads=shape.n_heads, n_kv_heads=shape.n_kv_heads,
                               head_dim=shape.head_dim, ffn=shape.ffn, vocab=shape.vocab,
                               mask_id=shape.mask_id, dtype=shape.dtype, qkv_bias=shape.qkv_bias,
                               rms_eps=shape.rms_eps, rope_theta=shape.rope_theta,
                               weight_fp8=fp8)
    m = wd.wd_init_model(cfg(False), ts, device)
    m8 = wd.wd_init_model(cfg(True), ts, device) if fp8_too else None
    del ts
    torch.cuda.empty_cache()
    return (m, m8) if fp8_too else m


def fp8_weight_variant(model8, prompts, w, n_steps, fixed_s):
    """The FP8-weight variant (not the paper's precision): the same windowed
    generation with e4m3 projection weights, steps/s and the roofline of its
    few-row GEMMs."""
    import paper_2601_20332_amd as wd
    import torch
    win = w.window
    wc = wd.window_config(win.n_active, win.n_buffer, win.refresh_every, win.unmask_per_step)
    generation(model8, prompts, w.gen_len, wc, n_steps)  # warm
    torch.cuda.synchronize()
    reps = 2
    t0 = time.perf_counter()
    for _ in range(reps):
        generation(model8, prompts, w.gen_len, wc, n_steps)
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / reps
    wd.wd_profile_enable(model8, True)
    t1 = time.perf_counter()
    generation(model8, prompts, w.gen_len, wc, n_steps)
    torch.cuda.synchronize()
    roof = roofline_of(model8, wd.WD_PROF_GEMM_ROWS, time.perf_counter() - t1)
    wd.wd_profile_enable(model8, False)
    if roof:
        roof["traffic"] = None  # the counter runs cover the bf16 kernels only
    return {
        "variant": "fp8 (e4m3) projection weights with per-row scales (not the paper's precision)",
        "steps_per_s": round(n_steps / t, 3),
        "ms_per_generation": round(t * 1e3, 2),
        "speedup_vs_bf16": round(fixed_s / t, 3),
        "roofline": roof,
    }


def other_workload(name: str, device: str, model=None, reps: int = 2, warm: bool = True,
                   full: bool = True):
    """Windowed generation on another workload: one model upload (or `model`,
    already packed, when the workload has the same model shape), one warm-up
    (`warm`), `reps` timed generations, one full-sequence generation for the
    speedup (`full`), one instrumented generation for the kernel rooflines."""
    import paper_2601_20332_amd as wd
    import synth
    import torch
    w = synth.WORKLOADS[name]
    own = model is None
    if own:
        t0 = time.time()
        model = upload_model(w.model, device)
        log(f"[bench] {name}: weights generated and packed in {time.time() - t0:.1f}s")
    prompts = synth.prompts(w.model, synth.prompt_lengths(w))
    win = w.window
    wc = wd.window_config(win.n_active, win.n_buffer, win.refresh_every, win.unmask_per_step)
    n_steps = len(wd.wd_plan(w.prompt_len, w.gen_len, wc)["n_rows"])
    if warm:
        generation(model, prompts, w.gen_len, wc, n_steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(reps):
        generation(model, prompts, w.gen_len, wc, n_steps, progress=128)
    torch.cuda.synchronize()
    t = (time.perf_counter() - t1) / reps
    log(f"[bench] {name}: {reps} timed generations, {t:.3f}s each")
    t_full = None
    if full:
        tf = time.perf_counter()
        generation(model, prompts, w.gen_len, wc, n_steps, full=True, progress=128)
        torch.cuda.synchronize()
        t_full = time.perf_counter() - tf
        log(f"[bench] {name}: full-sequence generation {t_full:.3f}s")
    wd.wd_profile_enable(model, True)
    te = time.perf_counter()
    generation(model, prompts, w.gen_len, wc, n_steps, progress=128)
    torch.cuda.synchronize()
    te = time.perf_counter() - te
    rows = roofline_of(model, wd.WD_PROF_GEMM_ROWS, te)
    tiled = roofline_of(model, wd.WD_PROF_GEMM_TILED, te)
    attn = roofline_of(model, wd.WD_PROF_ATTN, te)
    wd.wd_profile_enable(model, False)
    if own:
        model.free()
    for r in (rows, tiled, attn):
        if r:
            r["traffic"] = None  # the counter runs cover the LLaDA-8B workload
    B = len(prompts)
    m = w.model
    return {
        "workload": (f"{name}: {m.n_layers}L hidden {m.hidden} {m.n_heads}q/{m.n_kv_heads}kv x "
                     f"{m.head_dim} ffn {m.ffn} vocab {m.vocab}{' qkv bias' if m.qkv_bias else ''}, "
                     f"random init N(0,0.02)"),
        "batch": B, "prompt_len": w.prompt_len if B == 1 else synth.prompt_lengths(w),
        "gen_len": w.gen_len,
        "n_active": win.n_active, "n_buffer": win.n_buffer, "refresh_every": win.refresh_every,
        "unmask_per_step": win.unmask_per_step,
        "timed_generations": reps,
        "steps_per_s": round(n_steps / t, 3),
        "decoded_tokens_per_s": round(B * w.gen_len / t, 3),
        "ms_per_generation": round(t * 1e3, 2),
        "speedup_vs_full_sequence": round(t_full / t, 3) if t_full else None,
        "roofline": rows,
        "roofline_tiled_gemm": tiled,
        "roofline_attention": attn,
    }


def generation(model, prompts, G, wc, n_steps, full=False, progress=None):
    """One whole generation; with progress, a log line every `progress` steps
    (long full-sequence runs)."""
    import paper_2601_20332_amd as wd
    gen = wd.wd_prefill_prompt(model, prompts, G, wc)
    fn = wd.lib.wd_full_step if full else wd.lib.wd_step
    for i in range(n_steps):
        wd._check(fn(gen.handle, None))
        if progress and (i + 1) % progress == 0:
            log(f"[bench] {'full-sequence' if full else 'windowed'} step {i + 1}/{n_steps}")
    # synchronizes; raises if the device's checks of any step against the
    # host's schedule failed, so a generation that went wrong gives no record
    _, decoded, t = wd.wd_get_state(gen)
    gen.free()
    if t != n_steps or not all(d.all() for d in decoded):
        raise RuntimeError(f"generation ended after {t} steps with undecoded positions")


def run_until_done(model, prompts, G, wc):
    """One generation stepped until the library reports it finished; returns
    (steps taken, seconds, live ends)."""
    import paper_2601_20332_amd as wd
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    gen = wd.wd_prefill_prompt(model, prompts, G, wc)
    n = 0
    while True:
        st = wd.lib.wd_step(gen.handle, None)
        if st == wd.WD_ERR_STATE:
            break
        wd._check(st)
        n += 1
    ends = [int(e) for e in wd.wd_seq_ends(gen)]
    wd.wd_get_state(gen)  # raises if the device's checks failed
    gen.free()
    return n, time.perf_counter() - t0, ends


def adaptive_termination(model, prompts, w, n_steps, fixed_s):
    """Adaptive termination at <eos> (Sec. 4.2) on the same workload.  Random
    weights never aim at an <eos>, so the <eos> id is the token the fixed-length
    generation first decodes a quarter of the way through: with it as <eos>
    the generation ends there.  Also timed: the same tracked path with an id
    the generation never decodes (no early end), which isolates the cost of
    reading each step's decisions back."""
    import numpy as np
    import paper_2601_20332_amd as wd
    win = w.window
    plain = wd.window_config(win.n_active, win.n_buffer, win.refresh_every, win.unmask_per_step)
    gen = wd.wd_prefill_prompt(model, prompts, w.gen_len, plain)
    seen, eos, eos_step = set(), None, None
    for t in range(n_steps):
        r = wd.wd_step(gen, want_result=True)
        toks = [int(x) for x in r.tokens[0] if x >= 0]
        fresh = [x for x in toks if x not in seen]
        if eos is None and t >= n_steps // 4 and fresh:
            eos, eos_step = fresh[0], t
        seen.update(toks)
    final = wd.wd_get_state(gen)[0]
    gen.free()
    used = set(np.concatenate(final).tolist())
    unused = next(v for v in range(w.model.vocab - 1) if v not in used)

    def timed(eos_id, reps=2):
        wc = wd.window_config(win.n_active, win.n_buffer, win.refresh_every,
                              win.unmask_per_step, eos_id=eos_id)
        run_until_done(model, prompts, w.gen_len, wc)  # warm
        runs = [run_until_done(model, prompts, w.gen_len, wc) for _ in range(reps)]
        return runs[0][0], sum(r[1] for r in runs) / reps, runs[0][2]

    n_eos, t_eos, ends = timed(eos)
    n_none, t_none, _ = timed(unused)
    return {
        "eos_token": eos,
        "eos_first_decoded_at_step": eos_step,
        "live_end": ends,
        "seq_len": [len(p) + w.gen_len for p in prompts],
        "steps": n_eos,
        "fixed_length_steps": n_steps,
        "ms_per_generation": round(t_eos * 1e3, 2),
        "fixed_length_ms_per_generation": round(fixed_s * 1e3, 2),
        "speedup_vs_fixed_length": round(fixed_s / t_eos, 3),
        "tracked_no_eos_ms_per_generation": round(t_none * 1e3, 2),
        "tracking_overhead": round(t_none / fixed_s - 1.0, 4),
    }


def buffer_refresh_variant(model, prompts, w, n_steps, fixed_s):
    """The buffer-only refresh variant (not the paper's method) on the same
    workload: steps/s and the rows its later refreshes run."""
    import paper_2601_20332_amd as wd
    win = w.window
    wc = wd.window_config(win.n_active, win.n_buffer, win.refresh_every, win.unmask_per_step,
                          buffer_refresh=True)
    plan = wd.wd_plan(w.prompt_len, w.gen_len, wc)
    refresh_rows = [int(r) for r, f in zip(plan["n_rows"], plan["is_refresh"]) if f]
    generation(model, prompts, w.gen_len, wc, n_steps)  # warm
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    reps = 2
    for _ in range(reps):
        generation(model, prompts, w.gen_len, wc, n_steps)
    torch.cuda.synchronize()
    t = (time.perf_counter() - t0) / reps
    return {
        "variant": "buffer-only refresh (not the paper's method)",
        "steps_per_s": round(n_steps / t, 3),
        "ms_per_generation": round(t * 1e3, 2),
        "speedup_vs_paper_refresh": round(fixed_s / t, 3),
        "refresh_rows_first": refresh_rows[0],
        "refresh_rows_later_mean": round(sum(refresh_rows[1:]) / max(1, len(refresh_rows) - 1), 1),
    }


def cpu_model() -> str:
    """The host CPU's model name (/proc/cpuinfo), or the platform's string."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, plan, L_s=4, reps=20, ref_reps=10):
    """The float64 oracle on a bounded sample of the workload: after one untimed
    refresh forward (first-touch of its buffers), the mean of `ref_reps` refresh
    forwards (the largest retained prefix of the generation) over L_s of the
    layers, and the mean of `reps` normal-step forwards (the average online row
    count) over the same layers and of `reps` LM head + confidence passes on the
    active rows.
    Scaled to the full depth and summed over the generation's schedule (cost per
    layer taken as linear in the rows)."""
    import numpy as np
    from threadpoolctl import threadpool_info
    import synth
    from oracle.model import OracleModel
    from oracle.sampler import confidence
    shape = synth.with_layers(w.model, L_s)
    om = OracleModel(synth.Weights(shape), cache_budget_bytes=64e9)
    for name, _, _ in synth.tensor_specs(shape):
        if name != "emb":
            om.w(name)                                    # weights resident before timing
    S = w.prompt_len + w.gen_len
    prompt = synth.prompts(shape, [w.prompt_len])[0]
    x = np.concatenate([prompt, np.full(w.gen_len, shape.mask_id)])
    c_ref = max(p.ctx_len for p in plan if p.refresh)
    normal = [p.n_online for p in plan if not p.refresh]
    m_norm = int(round(sum(normal) / max(1, len(normal))))
    n_act = w.window.n_active
    tw = time.perf_counter()
    om.forward(x[:c_ref])
    t0 = time.perf_counter()
    for _ in range(ref_reps):
        h, K, V = om.forward(x[:c_ref])
    t1 = time.perf_counter()
    cache = om.new_cache(S)
    for l in range(L_s):
        cache.K[l][:c_ref] = K[l]
        cache.V[l][:c_ref] = V[l]
    rows = list(range(w.prompt_len, w.prompt_len + m_norm))
    t2 = time.perf_counter()
    for _ in range(reps):
        om.forward_rows(x[rows], rows, cache, c_ref)
    t3 = time.perf_counter()
    for _ in range(reps):
        confidence(om.logits(h[:n_act]), shape.mask_id)
    t4 = time.perf_counter()
    per_row_ref = (t1 - t0) / ref_reps / L_s / c_ref
    per_row_norm = (t3 - t2) / reps / L_s / m_norm
    head = (t4 - t3) / reps
    L = w.model.n_layers
    total = sum(L * (per_row_ref * p.n_online if p.refresh else per_row_norm * p.n_online) + head
                for p in plan)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {
        "value": len(plan) / total,
        "unit": "steps/s",
        "cores": int(threads),
        "cpu_model": cpu_model(),
        "host_cpus_available": len(os.sched_getaffinity(0)),
        "kind": "oracle",
        "sample": (f"float64 oracle, {L_s} of {L} layers: refresh forward over {c_ref} rows "
                   f"({(t1 - t0) / ref_reps:.1f} s, mean of {ref_reps}), normal-step forward over {m_norm} rows "
                   f"({(t3 - t2) / reps:.3f} s, mean of {reps}), LM head + confidence on {n_act} "
                   f"rows ({head:.3f} s, mean of {reps}); {t4 - tw:.1f} s in all with a warm-up forward; scaled to {L} "
                   f"layers and the {len(plan)}-step schedule (extrapolated)"),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3, help="timed whole generations")
    ap.add_argument("--warmup", type=int, default=1, help="untimed whole generations")
    ap.add_argument("--workload", default="llada8b",
                    choices=["llada8b", "dream7b", "llada8b_long", "llada8b_batch16"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-full", action="store_true", help="skip the full-sequence comparison")
    ap.add_argument("--full-once", action="store_true",
                    help="time the full-sequence generation without a warm-up run of its own "
                         "(the kernels are warm from the windowed runs)")
    ap.add_argument("--no-eos", action="store_true",
                    help="skip the adaptive-termination measurement")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the buffer-only refresh variant")
    ap.add_argument("--no-others", action="store_true",
                    help="skip the second workload shape (Dream-7B) and the peak probe")
    ap.add_argument("--no-events", action="store_true",
                    help="time without the per-launch GEMM events (no roofline)")
    ap.add_argument("--calibrate-copy", type=int, metavar="MIB", default=0,
                    help="only run 4 plain device-to-device copies of MIB MiB (the reference "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes) and exit")
    ap.add_argument("--pmc-summary", nargs=4, metavar=("GEMM_FETCH", "GEMM_WRITE", "COPY_FETCH",
                                                        "COPY_WRITE"),
                    help="only turn four rocprofv3 --pmc csv folders into HBM bytes per GEMM "
                         "launch and per layer of attention (copies of --calibrate-copy MiB, "
                         "default 1024), write profiles/kernel_traffic.json and exit; needs "
                         "no GPU")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, copy_mib=args.calibrate_copy or 1024)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the windowed step of one batch runs on one MI355X "
              "(no multi-GPU path is built); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        a = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(4):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_dispatch": n, "dispatches": 4}), flush=True)
        return
    import synth
    import paper_2601_20332_amd as wd

    w = synth.WORKLOADS[args.workload]
    device = "cuda:0"
    torch.cuda.set_device(0)
    t0 = time.time()
    want_fp8 = not args.no_variants and len(synth.prompt_lengths(w)) == 1
    if want_fp8:
        model, model8 = upload_model(w.model, device, fp8_too=True)
    else:
        model, model8 = upload_model(w.model, device), None
    log(f"[bench] {args.workload}: weights generated and packed in {time.time() - t0:.1f}s")
    prompts = synth.prompts(w.model, synth.prompt_lengths(w))
    win = w.window
    wc = wd.window_config(win.n_active, win.n_buffer, win.refresh_every, win.unmask_per_step)
    n_steps = len(wd.wd_plan(w.prompt_len, w.gen_len, wc)["n_rows"])

    for i in range(args.warmup):
        generation(model, prompts, w.gen_len, wc, n_steps)
        log(f"[bench] warmup generation {i + 1}/{args.warmup} done")

    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        generation(model, prompts, w.gen_len, wc, n_steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    log(f"[bench] {args.steps} timed generations in {elapsed:.3f}s")

    # Roofline of the dominant kernel: the same generations again, now with a
    # HIP event pair around every projection-GEMM launch on the library's stream
    # (kept out of the pass above, whose clock gives `value`).
    roofline = roofline_tiled = roofline_attn = None
    if not args.no_events:
        wd.wd_profile_enable(model, True)
        torch.cuda.synchronize()
        t_ev = time.perf_counter()
        for i in range(args.steps):
            generation(model, prompts, w.gen_len, wc, n_steps)
        torch.cuda.synchronize()
        elapsed_ev = time.perf_counter() - t_ev
        # the dominant kernel: few-row weight-streaming GEMM of the normal steps
        roofline = roofline_of(model, wd.WD_PROF_GEMM_ROWS, elapsed_ev)
        # second: the many-row GEMM of the refresh steps
        roofline_tiled = roofline_of(model, wd.WD_PROF_GEMM_TILED, elapsed_ev)
        # attention: K/V of [0, c) streamed per layer and step
        roofline_attn = roofline_of(model, wd.WD_PROF_ATTN, elapsed_ev)
        wd.wd_profile_enable(model, False)
        if roofline:
            roofline["instrumented_pass_s"] = round(elapsed_ev, 3)
        if args.workload != "llada8b":
            for r in (roofline, roofline_tiled, roofline_attn):
                if r:
                    r["traffic"] = None  # the counter runs cover the LLaDA-8B workload

    full_speedup = None
    if not args.no_full:
        if not args.full_once:
            generation(model, prompts, w.gen_len, wc, n_steps, full=True)  # warm
        torch.cuda.synchronize()
        tf = time.perf_counter()
        generation(model, prompts, w.gen_len, wc, n_steps, full=True, progress=64)
        torch.cuda.synchronize()
        t_full = time.perf_counter() - tf
        full_speedup = round(t_full / (elapsed / args.steps), 3)
        log(f"[bench] full-sequence generation {t_full:.3f}s")
    variant = fp8 = None
    if not args.no_variants and len(prompts) == 1:
        variant = buffer_refresh_variant(model, prompts, w, n_steps, elapsed / args.steps)
        log(f"[bench] buffer-only refresh variant: {variant}")
    if model8 is not None:
        fp8 = fp8_weight_variant(model8, prompts, w, n_steps, elapsed / args.steps)
        log(f"[bench] fp8-weight variant: {fp8}")
        model8.free()
    adaptive = None
    if not args.no_eos:
        adaptive = adaptive_termination(model, prompts, w, n_steps, elapsed / args.steps)
        log(f"[bench] adaptive termination: {adaptive}")
    peaks = None
    if not args.no_others:
        tf_meas, gbs_meas = wd.wd_measure_peaks(model)
        peaks = {"mfma_bf16_tflops": round(tf_meas, 1), "hbm_read_gbs": round(gbs_meas, 1),
                 "method": "independent 32x32x16 bf16 MFMAs on every CU; one non-temporal "
                           "read pass over 4 GiB"}
        log(f"[bench] measured peaks: {peaks}")
        for r in (roofline, roofline_tiled, roofline_attn):
            if r:
                meas = gbs_meas if r["unit"] == "GB/s" else tf_meas
                r["frac_of_measured_peak"] = round(r["achieved"] / meas, 4)
    others = None
    if not args.no_others and args.workload == "llada8b":
        others = {}
        # the same LLaDA-8B model: the long generation (Sec. 5.3, time against
        # generation length), with its full-sequence comparison, and the
        # ragged batch of 16 (windowed only: its full-sequence leg alone takes
        # about two minutes)
        others["llada8b_long"] = other_workload("llada8b_long", device, model=model, reps=2,
                                                warm=False)
        log(f"[bench] llada8b_long: {others['llada8b_long']}")
        others["llada8b_batch16"] = other_workload("llada8b_batch16", device, model=model, reps=1,
                                                   warm=False, full=False)
        log(f"[bench] llada8b_batch16: {others['llada8b_batch16']}")
    model.free()
    if others is not None:
        others["dream7b"] = other_workload("dream7b", device)
        log(f"[bench] dream7b: {others['dream7b']}")
        if peaks:
            for o in others.values():
                for r in (o["roofline"], o["roofline_tiled_gemm"], o["roofline_attention"]):
                    if r:
                        meas = peaks["hbm_read_gbs"] if r["unit"] == "GB/s" else peaks["mfma_bf16_tflops"]
                        r["frac_of_measured_peak"] = round(r["achieved"] / meas, 4)

    cpu = None
    if not args.no_cpu_baseline:
        from oracle.schedule import plan_counts
        plan = plan_counts(w.prompt_len, w.gen_len, win)
        cpu = cpu_baseline(w, plan)
        log(f"[bench] cpu baseline: {cpu}")

    B = len(prompts)
    steps_per_s = args.steps * n_steps / elapsed
    out = {
        "metric": METRIC,
        "value": round(steps_per_s, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"{args.workload}: {w.model.n_layers}L hidden {w.model.hidden} "
                         f"{w.model.n_heads}q/{w.model.n_kv_heads}kv x {w.model.head_dim} "
                         f"ffn {w.model.ffn} vocab {w.model.vocab}, random init N(0,0.02)"),
            "batch": B,
            "prompt_len": w.prompt_len,
            "gen_len": w.gen_len,
            "n_active": win.n_active,
            "n_buffer": win.n_buffer,
            "refresh_every": win.refresh_every,
            "unmask_per_step": win.unmask_per_step,
            "bench_step": f"one whole generation = {n_steps} denoising steps",
        },
        "decoded_tokens_per_s": round(args.steps * B * w.gen_len / elapsed, 3),
        "speedup_vs_full_sequence": full_speedup,
        "roofline": roofline,
        "roofline_tiled_gemm": roofline_tiled,
        "roofline_attention": roofline_attn,
        "adaptive_termination": adaptive,
        "buffer_refresh_variant": variant,
        "fp8_weight_variant": fp8,
        "measured_peaks": peaks,
        "other_workloads": others,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
