"""Pins of the oracle's windowed schedule (Secs. 4.2-4.3): a hand-derived
walk-through, closed-form counts, set invariants, the full-equivalence and
truncation special cases, cache consistency, pruning and resume."""
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import synth
from oracle.model import KVCache, OracleModel
from oracle.schedule import (FullDecoder, WindowedDecoder, generate_full, generate_windowed,
                             plan_counts)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "window_walkthrough.txt")


class StubModel:
    """Random logits, no network: exercises only the schedule's bookkeeping."""

    def __init__(self, vocab=24, seed=0):
        self.shape = synth.ModelShape(n_layers=1, hidden=2, n_heads=1, n_kv_heads=1, head_dim=2,
                                      ffn=2, vocab=vocab, dtype=synth.DTYPE_F32)
        self.rng = np.random.default_rng(seed)
        self.rows_seen = []

    def forward(self, ids, positions=None):
        n = len(ids)
        self.rows_seen.append(list(range(n)))
        return np.zeros((n, 2)), [np.zeros((n, 1, 2))], [np.zeros((n, 1, 2))]

    def forward_rows(self, ids, pos, cache, ctx):
        assert max(pos) < ctx
        self.rows_seen.append(list(pos))
        return np.zeros((len(ids), 2))

    def logits(self, h):
        return self.rng.standard_normal((h.shape[0], self.shape.vocab))

    def new_cache(self, S):
        return KVCache(1, S, 1, 2)


def micro(dtype=synth.DTYPE_F32, n_kv=2, seed=3):
    shape = synth.ModelShape(n_layers=2, hidden=32, n_heads=4, n_kv_heads=n_kv, head_dim=8,
                             ffn=48, vocab=64, dtype=dtype, qkv_bias=True, rope_theta=100.0)
    return OracleModel(synth.Weights(shape, seed=seed, std=0.3))


def rightmost(k):
    def pick(rec):
        sel = sorted(rec.active)[::-1][:k]
        return sel, {p: 1 for p in sel}
    return pick


def _parse_set(s, ctx=None):
    if s == "-":
        return []
    if ".." in s:
        a, b = s.split("..")
        return list(range(int(a), int(b) + 1))
    return [int(v) for v in s.split(",")]


def load_golden():
    cases, cur = [], None
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        if f[0] == "case":
            cur = {"name": f[1], "args": [int(v) for v in f[2:]], "rows": []}
        elif f[0] == "end":
            cases.append(cur)
        else:
            cur["rows"].append(f)
    return cases


@pytest.mark.parametrize("case", load_golden(), ids=lambda c: c["name"])
def test_hand_walkthrough(case):
    n_p, G, na, nb, R, k = case["args"]
    win = synth.WindowSettings(na, nb, R, k)
    m = StubModel()
    dec = WindowedDecoder(m, list(range(n_p)), G, win)
    for row in case["rows"]:
        t, refresh, ctx = int(row[0]), bool(int(row[1])), int(row[2])
        rec = dec.step(override=rightmost(k))
        assert rec.t == t and rec.refresh == refresh and rec.ctx_len == ctx
        assert rec.window == _parse_set(row[3])
        assert rec.active == _parse_set(row[4])
        assert sorted(rec.phase_decoded) == _parse_set(row[5])
        buf = [p for p in rec.window if p not in rec.active and p not in rec.phase_decoded]
        assert buf == _parse_set(row[6])
        assert rec.online == _parse_set(row[7])
        assert rec.selected == _parse_set(row[8])
    assert dec.done()
    plan = plan_counts(n_p, G, win)
    assert len(plan) == len(case["rows"])


settings_small = settings(max_examples=120, deadline=None)


@settings_small
@given(n_p=st.integers(1, 12), G=st.integers(1, 60), na=st.integers(1, 9),
       nb=st.integers(0, 12), R=st.integers(1, 9), k=st.integers(1, 4), seed=st.integers(0, 99))
@pytest.mark.parametrize("refresh", ["full", "buffer"])
def test_counts_closed_form_and_invariants(n_p, G, na, nb, R, k, seed, refresh):
    """plan_counts (counts only) equals the trajectory's counts for any decode
    order; roles partition W_ex; the active window only moves right; no
    far-field position is ever computed."""
    win = synth.WindowSettings(na, nb, R, k)
    m = StubModel(seed=seed)
    dec = WindowedDecoder(m, list(range(n_p)), G, win, refresh=refresh)
    plan = plan_counts(n_p, G, win, refresh=refresh)
    recs = []
    prev_active = None
    while not dec.done():
        und_before = set(np.flatnonzero(~dec.decoded).tolist())
        rec = dec.step()
        recs.append(rec)
        W = set(rec.window)
        A, Dp = set(rec.active), set(rec.phase_decoded)
        B = W - A - Dp
        assert A | Dp | B == W and not (A & Dp) and not (A & B) and not (Dp & B)
        assert all(p < rec.ctx_len for p in rec.online)
        assert all(p in und_before for p in A)
        if rec.refresh:
            und = sorted(und_before)
            assert rec.window == und[:win.external]
            assert rec.ctx_len == (und[win.external - 1] + 1 if len(und) >= win.external
                                   else n_p + G)
            # [0, c) is exactly the decoded positions plus W_ex
            dec_pos = {p for p in range(n_p + G) if p not in und_before}
            assert set(range(rec.ctx_len)) == (dec_pos & set(range(rec.ctx_len))) | W
            assert all(p < rec.ctx_len for p in dec_pos)
        else:
            # monotone window: no undecoded member is lost, the minimum never decreases
            still = prev_active - set(recs[-2].selected)
            assert still <= A
            if A and still:
                assert min(A) >= min(still)
        prev_active = A
        assert m.rows_seen[-1] == rec.online
    assert len(recs) == len(plan)
    for rec, p in zip(recs, plan):
        assert rec.refresh == p.refresh and rec.ctx_len == p.ctx_len
        assert len(rec.active) == p.n_active and len(rec.online) == p.n_online
        assert len(rec.phase_decoded) == p.n_phase_decoded and len(rec.selected) == p.n_decode
    ctxs = [r.ctx_len for r in recs]
    assert ctxs == sorted(ctxs)


def test_counts_of_the_benchmark_workloads():
    """With k decodes every step, c_p = min(S, n_p + k R p + E) and
    |O| = |A| + k j (j = step within the phase)."""
    for name, w in synth.WORKLOADS.items():
        if w.ragged_prompt:
            continue
        win = w.window
        plan = plan_counts(w.prompt_len, w.gen_len, win)
        S = w.prompt_len + w.gen_len
        k, R = win.unmask_per_step, win.refresh_every
        assert len(plan) == -(-w.gen_len // k)
        for t, p in enumerate(plan):
            ph, j = divmod(t, R)
            assert p.refresh == (j == 0)
            assert p.ctx_len == min(S, w.prompt_len + k * R * ph + win.external)
            if not p.refresh:
                assert p.n_online == p.n_active + k * j


@pytest.mark.parametrize("dtype", [synth.DTYPE_F32, synth.DTYPE_BF16])
def test_full_equivalence(dtype):
    """E >= G, n_act >= G and R = 1: Window-Diffusion is standard decoding."""
    m = micro(dtype)
    prompt = [5, 9, 2, 40, 17]
    G, k = 9, 2
    xw, rw = generate_windowed(m, prompt, G, synth.WindowSettings(G, 0, 1, k), keep_logits=True)
    xf, rf = generate_full(m, prompt, G, k, keep_logits=True)
    np.testing.assert_array_equal(xw, xf)
    assert [r.selected for r in rw] == [r.selected for r in rf]
    for a, b in zip(rw, rf):
        assert a.active == b.active
        np.testing.assert_array_equal(a.logits, b.logits)


def test_truncation_only_equals_forward_on_prefix():
    """R = 1: every step is the forward over the retained prefix [0, c)."""
    m = micro()
    prompt = [1, 2, 3, 4]
    G = 12
    win = synth.WindowSettings(2, 3, 1, 1)
    dec = WindowedDecoder(m, prompt, G, win)
    while not dec.done():
        x = dec.x.copy()
        und = np.flatnonzero(~dec.decoded)
        c = und[win.external - 1] + 1 if len(und) >= win.external else len(x)
        A = [int(p) for p in und[:win.n_active] if p < c]
        h, _, _ = m.forward(x[:c])
        want = m.logits(h[A])
        rec = dec.step(keep_logits=True)
        assert rec.refresh and rec.ctx_len == c and rec.active == A
        np.testing.assert_array_equal(rec.logits, want)


@pytest.mark.parametrize("dtype", [synth.DTYPE_F32, synth.DTYPE_BF16])
def test_refresh_cache_matches_fresh_forward(dtype):
    m = micro(dtype, n_kv=1)
    mask = m.shape.mask_id
    dec = WindowedDecoder(m, [7, 8, 9], 20, synth.WindowSettings(3, 4, 3, 2))
    seen = 0
    while not dec.done():
        before = dec.x.copy()
        rec = dec.step()
        if rec.refresh:
            seen += 1
            c = rec.ctx_len
            _, K, V = m.forward(before[:c])
            for l in range(m.shape.n_layers):
                np.testing.assert_array_equal(dec.cache.K[l][:c], K[l])
                np.testing.assert_array_equal(dec.cache.V[l][:c], V[l])
            assert all(before[p] == mask for p in rec.active)
    assert seen >= 3


@pytest.mark.parametrize("dtype", [synth.DTYPE_F32, synth.DTYPE_BF16])
def test_rows_over_fresh_cache_reproduce_refresh(dtype):
    """I4: right after a refresh, recomputing any row subset online (its K/V
    overwrite identical values) reproduces the refresh's hidden states."""
    m = micro(dtype)
    rng = np.random.default_rng(0)
    ids = rng.integers(0, m.shape.vocab - 1, size=14)
    c = 11
    h, K, V = m.forward(ids[:c])
    for trial in range(4):
        cache = m.new_cache(14)
        for l in range(m.shape.n_layers):
            cache.K[l][:c] = K[l]
            cache.V[l][:c] = V[l]
        rows = sorted(rng.choice(c, size=rng.integers(1, c), replace=False).tolist())
        hr = m.forward_rows(ids[rows], rows, cache, c)
        np.testing.assert_allclose(hr, h[rows], rtol=1e-10, atol=1e-10)


def test_far_field_is_pruned():
    """I5: tokens after c and cache rows at or after c never influence a step."""
    m = micro()
    G = 16
    win = synth.WindowSettings(2, 3, 3, 1)
    ref = WindowedDecoder(m, [3, 4], G, win)
    alt = WindowedDecoder(m, [3, 4], G, win)
    rng = np.random.default_rng(9)
    while not ref.done():
        a = ref.step(keep_logits=True)
        # scramble the far field of alt and poison its cache beyond c
        c = a.ctx_len
        if c < alt.S:
            keep = alt.x.copy()
            alt.x[c:] = rng.integers(0, m.shape.vocab, size=alt.S - c)
            for l in range(m.shape.n_layers):
                alt.cache.K[l][c:] = np.nan
                alt.cache.V[l][c:] = np.nan
        b = alt.step(keep_logits=True)
        if c < alt.S:
            alt.x[c:] = np.where(alt.decoded[c:], alt.x[c:], keep[c:])
        assert a.refresh == b.refresh and a.online == b.online
        np.testing.assert_array_equal(a.logits, b.logits)
        assert all(p < c for p in a.active + a.online)
        assert np.isfinite(a.logits).all()


def test_resume_at_phase_boundary():
    """I9: (x, decoded, t) at a phase start is the whole state."""
    m = micro()
    win = synth.WindowSettings(2, 2, 3, 1)
    full = WindowedDecoder(m, [1, 2, 3], 12, win)
    recs = [full.step() for _ in range(6)]
    x_mid = full.x.copy()
    dec_mid = full.decoded.copy()
    tail = []
    while not full.done():
        tail.append(full.step())
    res = WindowedDecoder(m, [1, 2, 3], 12, win)
    res.x[:] = x_mid
    res.decoded[:] = dec_mid
    res.t = 6
    tail2 = []
    while not res.done():
        tail2.append(res.step())
    assert [r.selected for r in tail] == [r.selected for r in tail2]
    np.testing.assert_array_equal(full.x, res.x)
    assert recs[0].refresh and tail[0].refresh


def test_full_decoder_candidates_are_all_masked():
    m = micro()
    dec = FullDecoder(m, [1, 2], 6, 2)
    rec = dec.step()
    assert rec.active == list(range(2, 8)) and len(rec.selected) == 2


# ---- adaptive termination at <eos> -------------------------------------------------------

EOS_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "eos_walkthrough.txt")
EOS = 5   # <eos> id of the walk-throughs (StubModel vocabulary of 24)


def load_eos_golden():
    cases, cur = [], None
    for line in open(EOS_GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        if f[0] == "case":
            cur = {"name": f[1], "args": [int(v) for v in f[2:8]],
                   "eos_steps": [int(v) for v in f[8].split(",")], "rows": []}
        elif f[0] == "end":
            cases.append(cur)
        else:
            cur["rows"].append(f)
    return cases


def rightmost_with_eos(k, eos_steps, eos=EOS):
    def pick(rec):
        sel = sorted(rec.active)[::-1][:k]
        toks = {p: 1 for p in sel}
        if rec.t in eos_steps and sel:
            toks[sel[0]] = eos
        return sel, toks
    return pick


@pytest.mark.parametrize("case", load_eos_golden(), ids=lambda c: c["name"])
def test_eos_hand_walkthrough(case):
    n_p, G, na, nb, R, k = case["args"]
    win = synth.WindowSettings(na, nb, R, k)
    dec = WindowedDecoder(StubModel(), list(range(n_p)), G, win, eos_id=EOS)
    pick = rightmost_with_eos(k, case["eos_steps"])
    for row in case["rows"]:
        t, refresh, ctx = int(row[0]), bool(int(row[1])), int(row[2])
        assert not dec.done()
        rec = dec.step(override=pick)
        assert rec.t == t and rec.refresh == refresh and rec.ctx_len == ctx
        assert rec.window == _parse_set(row[3])
        assert rec.active == _parse_set(row[4])
        assert sorted(rec.phase_decoded) == _parse_set(row[5])
        buf = [p for p in rec.window
               if p not in rec.active and p not in rec.phase_decoded and p < ctx]
        assert buf == _parse_set(row[6])
        assert rec.online == _parse_set(row[7])
        assert rec.selected == _parse_set(row[8])
    assert dec.done()
    # past the end only tokens decoded before the end moved there remain; every
    # other position keeps the mask token
    past = dec.decoded[dec.end:]
    assert (dec.x[dec.end:][~past] == dec.model.shape.mask_id).all()
    assert past.sum() == (1 if case["name"] == "F" else 0)


@settings_small
@given(n_p=st.integers(1, 10), G=st.integers(1, 40), na=st.integers(1, 8),
       nb=st.integers(0, 10), R=st.integers(1, 8), k=st.integers(1, 3), seed=st.integers(0, 99),
       eos_steps=st.sets(st.integers(0, 30), max_size=3))
def test_eos_invariants(n_p, G, na, nb, R, k, seed, eos_steps):
    """Whatever steps write <eos>: nothing at or after the end is ever computed
    again, the schedule finishes exactly the live prefix, and it never takes
    more steps than decoding without <eos>."""
    win = synth.WindowSettings(na, nb, R, k)
    rng = np.random.default_rng(seed)

    def pick(rec):
        n = min(k, len(rec.active))
        sel = [int(p) for p in rng.choice(rec.active, size=n, replace=False)]
        toks = {p: 1 for p in sel}
        if rec.t in eos_steps:
            toks[sel[int(rng.integers(len(sel)))]] = EOS
        return sel, toks

    dec = WindowedDecoder(StubModel(seed=seed), list(range(n_p)), G, win, eos_id=EOS)
    ends = []
    steps = 0
    while not dec.done():
        end_before = dec.end
        rec = dec.step(override=pick)
        steps += 1
        assert rec.ctx_len <= end_before
        assert all(p < end_before for p in rec.online)
        assert all(p < end_before for p in rec.active)
        assert all(p < end_before for p in rec.phase_decoded)
        if rec.refresh:
            assert rec.online == list(range(rec.ctx_len))
        ends.append(dec.end)
        assert steps <= G
    assert ends == sorted(ends, reverse=True)           # the end only moves forward
    assert dec.decoded[:dec.end].all()
    mask = dec.model.shape.mask_id
    assert (dec.x[dec.end:][~dec.decoded[dec.end:]] == mask).all()
    written = [p for p in range(n_p, dec.S) if dec.decoded[p] and dec.x[p] == EOS]
    assert dec.end == (min(written) + 1 if written else dec.S)
    plain = plan_counts(n_p, G, win)
    assert steps <= len(plain)
    if not written:
        assert steps == len(plain)


def test_eos_never_written_changes_nothing():
    m = micro()
    win = synth.WindowSettings(3, 4, 3, 2)
    prompt = [3, 9, 27, 1]
    # an id the trajectory never produces: the run equals the one without <eos>
    x0, r0 = generate_windowed(m, prompt, 14, win, keep_logits=True)
    unused = next(v for v in range(m.shape.vocab - 1) if v not in set(x0.tolist()))
    x1, r1 = generate_windowed(m, prompt, 14, win, keep_logits=True, eos_id=unused)
    assert (x0 == x1).all() and len(r0) == len(r1)
    for a, b in zip(r0, r1):
        assert a.online == b.online and a.ctx_len == b.ctx_len
        np.testing.assert_array_equal(a.logits, b.logits)


@pytest.mark.parametrize("eos_at", [0, 1, 2])
def test_eos_degenerate_windows_equal_adaptive_full_decoding(eos_at):
    """With W_ex covering every masked position, a refresh every step and
    every undecoded position active, the windowed decoder with <eos> is the
    plain adaptive-length full decoder: a full forward over [0, end) and every
    live masked position a candidate, at every step."""
    m = micro()
    prompt = [5, 17, 33]
    G, k = 10, 2
    win = synth.WindowSettings(G, 0, 1, k)
    eos = 7

    def inject(rec):
        toks = dict(rec.chosen_tokens)
        if rec.t == eos_at and rec.selected:
            toks[rec.selected[-1]] = eos
        return rec.selected, toks

    xw, rw = generate_windowed(m, prompt, G, win, override=inject, keep_logits=True, eos_id=eos)
    xf, rf = generate_full(m, prompt, G, k, override=inject, keep_logits=True, eos_id=eos)
    assert len(rw) == len(rf) and (xw == xf).all()
    for a, b in zip(rw, rf):
        assert a.active == b.active and a.ctx_len == b.ctx_len and a.selected == b.selected
        np.testing.assert_allclose(a.logits, b.logits, rtol=0, atol=1e-12)
    # the sequence ended before its last position, which was never decoded
    e = min(p for p in range(len(prompt), len(xw)) if xw[p] == eos)
    assert e < len(xw) - 1 and xw[-1] == m.shape.mask_id


# ---- buffer-only refresh (a variant, not the paper's method) -----------------------------

BUF_GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "buffer_refresh_walkthrough.txt")


def load_buffer_golden():
    global GOLDEN
    saved, GOLDEN = GOLDEN, BUF_GOLDEN
    try:
        return load_golden()
    finally:
        GOLDEN = saved


@pytest.mark.parametrize("case", load_buffer_golden(), ids=lambda c: c["name"])
def test_buffer_refresh_hand_walkthrough(case):
    n_p, G, na, nb, R, k = case["args"]
    win = synth.WindowSettings(na, nb, R, k)
    m = StubModel()
    dec = WindowedDecoder(m, list(range(n_p)), G, win, refresh="buffer")
    for row in case["rows"]:
        t, refresh, ctx = int(row[0]), bool(int(row[1])), int(row[2])
        rec = dec.step(override=rightmost(k))
        assert rec.t == t and rec.refresh == refresh and rec.ctx_len == ctx
        assert rec.window == _parse_set(row[3])
        assert rec.active == _parse_set(row[4])
        assert sorted(rec.phase_decoded) == _parse_set(row[5])
        assert rec.online == _parse_set(row[7])
        assert rec.selected == _parse_set(row[8])
        # the model saw exactly the online rows of the step
        assert m.rows_seen[-1] == rec.online
    assert dec.done()


def test_buffer_refresh_keeps_other_cache_rows_and_matches_full_first_phase():
    m = micro()
    win = synth.WindowSettings(3, 3, 3, 1)
    prompt = [4, 8, 15, 16, 23]
    G = 12
    full = WindowedDecoder(m, prompt, G, win)
    buf = WindowedDecoder(m, prompt, G, win, refresh="buffer")
    while not full.done():
        K_before = [k.copy() for k in buf.cache.K]
        rf = full.step(keep_logits=True)
        # the variant follows the same decisions, so both runs share one trajectory
        rb = buf.step(override=lambda rec: (rf.selected, rf.chosen_tokens), keep_logits=True)
        assert rb.active == rf.active
        if rb.t < win.refresh_every:
            # first phase: identical to the paper's refresh
            np.testing.assert_array_equal(rf.logits, rb.logits)
        if rb.refresh and rb.t > 0:
            assert rb.online == sorted(set(rb.window) | set(buf.prev_phase_decoded))
            untouched = [p for p in range(rb.ctx_len) if p not in rb.online]
            assert untouched, "some rows must keep their cache"
            for l in range(m.shape.n_layers):
                np.testing.assert_array_equal(buf.cache.K[l][untouched], K_before[l][untouched])
    assert buf.done()
