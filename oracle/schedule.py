"""Window-Diffusion's inference schedule (Secs. 4.1-4.3) and the standard
full-sequence decoding it approximates (Sec. 3.1), for one sequence.

State: the token sequence x of fixed length S = n_p + G (prompt, then G
[MASK] tokens) and the set of decoded positions (the prompt counts as
decoded).  Each diffusion step decodes up to k positions.

Window-Diffusion (Sec. 4.2, Sec. 4.3):

* Denoising is cut into phases; a phase is one refresh step followed by
  normal steps, R steps in all.
* At a phase start the external window W_ex is re-determined as a
  fixed-length prefix of the undecoded region: the first E undecoded
  positions in index order (all of them if fewer remain).  It stays fixed
  for the whole phase.  Undecoded positions after it are far-field and take
  no part in any computation of the phase.
* Because every decoded position lies before the E-th undecoded one (a
  position can only be decoded while inside a window), the tokens of the
  phase, D(<p) plus W_ex, are exactly the prefix [0, c) with
  c = (E-th undecoded position) + 1, or S when fewer than E remain.
* The internal window, the active set A(t), is the first n_active positions
  of W_ex that are still undecoded at step t.  Only A(t) gets logits.
* D_p(t) are the positions decoded so far inside the phase; the buffer is
  W_ex minus (A(t) union D_p(t)).
* Refresh step: a full forward over [0, c) whose K/V (every layer, every
  row) replace the cache (refresh equation of Sec. 4.3); the active rows'
  logits come from that same forward.
* Normal step: the online rows O = A(t) union D_p(t) run the full layer
  stack; their fresh K/V overwrite their cache rows and they attend to all
  of [0, c); buffer and pre-phase rows keep the refresh's K/V.  Tokens
  decoded inside the phase stay online until the next refresh
  (Sec. 4.3, and the refresh-cycle ablation of Sec. 5.3).

Adaptive termination (Sec. 4.2, adaptive termination; optional, eos_id):

* Once an <eos> token is decoded at a generated position e, the sequence
  ends at e: end = e + 1 (the first such position if there are several;
  end = S while none is decoded).  Positions at or after end are far-field
  for good: they leave the active set, the online rows and the attention
  context at once (the internal window stops advancing), and no later
  window reaches them.
* At a phase start W_ex and c are taken over [0, end) only: W_ex = the
  first E undecoded positions below end, c = (E-th of them) + 1, or end
  when fewer remain.  Within a phase the attention context is [0, min(c,
  end)).
* The sequence is finished when every position below end is decoded.  The
  positions after it keep the mask token.

Buffer-only refresh (a variant, not the paper's method; refresh="buffer"):

* The first phase refreshes [0, c) as above.  Every later refresh
  recomputes only the window W_ex and the positions decoded in the previous
  phase (D_{p-1}; the one decoded at a phase's last step still holds K/V
  computed from its [MASK] input), through the same online-row forward as a
  normal step; the other rows of [0, c) (the prompt and tokens decoded
  earlier) keep the K/V they were last given.

Readings where the paper is silent:

* A refresh happens at step 0 and then every R steps; a phase also ends
  early if its window has no undecoded position left while far-field
  positions remain (the next step then starts a new phase).
* The refresh step is itself a decoding step (logits on A at every step).
* Positions are absolute indices; batched sequences are independent.
* Only generated positions end a sequence: an <eos> id inside the prompt
  does not.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Dict, List, Optional, Sequence, Tuple

import numpy as np

import synth
from .model import OracleModel
from .sampler import confidence, select_updates


@dataclasses.dataclass
class StepRecord:
    t: int
    refresh: bool
    ctx_len: int                 # attended prefix [0, c) (min(c, end) with <eos>)
    window: List[int]            # W_ex of the current phase
    active: List[int]            # A(t)
    online: List[int]            # rows computed this step (= [0, c) on a refresh)
    phase_decoded: List[int]     # D_p(t) below end, before this step's update
    logits: Optional[np.ndarray]  # [|A|, V] (None unless kept)
    tokens: np.ndarray           # argmax candidate per active row
    conf: np.ndarray             # float32 confidence per active row
    selected: List[int]          # positions decoded this step, in rank order
    chosen_tokens: Dict[int, int]  # position -> token written


Override = Callable[[StepRecord], Optional[Tuple[List[int], Dict[int, int]]]]


def _apply_override(rec: StepRecord, override: Optional[Override]) -> None:
    if override is None:
        return
    res = override(rec)
    if res is not None:
        rec.selected, rec.chosen_tokens = list(res[0]), dict(res[1])


class _EosEnd:
    """The live end of a sequence under adaptive termination: one past the
    first generated position holding the <eos> token (S while there is none)."""

    eos_id: Optional[int]
    n_p: int
    end: int
    x: np.ndarray

    def _apply_eos(self, positions) -> None:
        if self.eos_id is None:
            return
        for p in positions:
            if p >= self.n_p and int(self.x[p]) == self.eos_id:
                self.end = min(self.end, int(p) + 1)


class WindowedDecoder(_EosEnd):
    """Window-Diffusion decoding of one sequence with the oracle model."""

    def __init__(self, model: OracleModel, prompt: Sequence[int], gen_len: int,
                 win: synth.WindowSettings, eos_id: Optional[int] = None,
                 refresh: str = "full"):
        if win.n_active < 1 or win.unmask_per_step < 1 or win.refresh_every < 1:
            raise ValueError("window settings must be positive")
        if win.n_buffer < 0 or gen_len < 1:
            raise ValueError("bad window or generation length")
        if refresh not in ("full", "buffer"):
            raise ValueError("refresh is 'full' (the paper's) or 'buffer' (variant)")
        self.model = model
        self.win = win
        self.eos_id = eos_id
        self.refresh_mode = refresh
        self.phases = 0                     # phases started so far
        self.prev_phase_decoded: List[int] = []
        self.n_p = len(prompt)
        self.S = self.n_p + gen_len
        self.end = self.S                   # live positions are [0, end)
        mask = model.shape.mask_id
        self.x = np.concatenate([np.asarray(prompt, dtype=np.int64),
                                 np.full(gen_len, mask, dtype=np.int64)])
        self.decoded = np.zeros(self.S, dtype=bool)
        self.decoded[:self.n_p] = True
        self.t = 0
        self.j: Optional[int] = None        # steps taken in the current phase
        self.window: List[int] = []
        self.ctx_len = 0
        self.phase_decoded: List[int] = []
        self.cache = model.new_cache(self.S)

    # -- bookkeeping -----------------------------------------------------
    def done(self) -> bool:
        return bool(self.decoded[:self.end].all())

    def needs_phase(self) -> bool:
        if self.j is None or self.j >= self.win.refresh_every:
            return True
        return not any(not self.decoded[i] and i < self.end for i in self.window)

    def slide(self) -> None:
        """Phase start: re-determine W_ex and the retained prefix [0, c)."""
        und = np.flatnonzero(~self.decoded[:self.end])
        E = self.win.external
        self.window = [int(i) for i in und[:E]]
        self.ctx_len = int(und[E - 1]) + 1 if len(und) >= E else self.end
        self.prev_phase_decoded = self.phase_decoded
        self.phase_decoded = []
        self.j = 0
        self.phases += 1

    def context(self) -> int:
        """Length of the attended prefix this step."""
        return min(self.ctx_len, self.end)

    def live_phase_decoded(self) -> List[int]:
        return [p for p in self.phase_decoded if p < self.end]

    def active(self) -> List[int]:
        und = [i for i in self.window if not self.decoded[i] and i < self.end]
        return und[:self.win.n_active]

    def online(self) -> List[int]:
        return sorted(set(self.active()) | set(self.live_phase_decoded()))

    def buffer(self) -> List[int]:
        a = set(self.active())
        d = set(self.phase_decoded)
        return [i for i in self.window if i not in a and i not in d and i < self.end]

    # -- one diffusion step ------------------------------------------------
    def step(self, override: Optional[Override] = None, keep_logits: bool = False) -> StepRecord:
        if self.done():
            raise RuntimeError("all positions are decoded")
        m = self.model
        refresh = self.needs_phase()
        if refresh:
            self.slide()
            c = self.ctx_len
            A = self.active()
            if self.refresh_mode == "buffer" and self.phases > 1:
                rows = sorted(set(self.window) |
                              {p for p in self.prev_phase_decoded if p < c})
                hR = m.forward_rows(self.x[rows], rows, self.cache, c)
                where = {p: i for i, p in enumerate(rows)}
                hA = hR[[where[p] for p in A]]
            else:
                h, Ks, Vs = m.forward(self.x[:c])
                for l in range(len(Ks)):
                    self.cache.K[l][:c] = Ks[l]
                    self.cache.V[l][:c] = Vs[l]
                rows = list(range(c))
                hA = h[A]
        else:
            A = self.active()
            rows = self.online()
            hO = m.forward_rows(self.x[rows], rows, self.cache, self.context())
            where = {p: i for i, p in enumerate(rows)}
            hA = hO[[where[p] for p in A]]
        logits = m.logits(hA)
        tok, conf = confidence(logits, m.shape.mask_id)
        sel = select_updates(A, conf, self.win.unmask_per_step)
        rec = StepRecord(t=self.t, refresh=refresh, ctx_len=self.context(),
                         window=list(self.window), active=list(A), online=rows,
                         phase_decoded=self.live_phase_decoded(),
                         logits=logits, tokens=tok, conf=conf, selected=sel,
                         chosen_tokens={p: int(tok[A.index(p)]) for p in sel})
        _apply_override(rec, override)
        for p in rec.selected:
            assert not self.decoded[p] and p in A
            self.x[p] = rec.chosen_tokens[p]
            self.decoded[p] = True
            self.phase_decoded.append(p)
        self._apply_eos(rec.selected)
        self.t += 1
        self.j += 1
        if not keep_logits:
            rec.logits = None
        return rec


class FullDecoder(_EosEnd):
    """Standard mask-based DLM decoding (Sec. 3.1): every step is a full forward
    over all S positions; every undecoded position is a candidate.  With
    eos_id, the forward and the candidates stop at the live end (the
    adaptive-length counterpart of the windowed decoder)."""

    def __init__(self, model: OracleModel, prompt: Sequence[int], gen_len: int, k: int,
                 eos_id: Optional[int] = None):
        self.model = model
        self.k = k
        self.eos_id = eos_id
        self.n_p = len(prompt)
        self.S = self.n_p + gen_len
        self.end = self.S
        self.x = np.concatenate([np.asarray(prompt, dtype=np.int64),
                                 np.full(gen_len, model.shape.mask_id, dtype=np.int64)])
        self.decoded = np.zeros(self.S, dtype=bool)
        self.decoded[:self.n_p] = True
        self.t = 0

    def done(self) -> bool:
        return bool(self.decoded[:self.end].all())

    def step(self, override: Optional[Override] = None, keep_logits: bool = False) -> StepRecord:
        m = self.model
        n = self.end
        h, _, _ = m.forward(self.x[:n])
        cand = [int(i) for i in np.flatnonzero(~self.decoded[:n])]
        logits = m.logits(h[cand])
        tok, conf = confidence(logits, m.shape.mask_id)
        sel = select_updates(cand, conf, self.k)
        rec = StepRecord(t=self.t, refresh=True, ctx_len=n, window=cand, active=cand,
                         online=list(range(n)), phase_decoded=[], logits=logits,
                         tokens=tok, conf=conf, selected=sel,
                         chosen_tokens={p: int(tok[cand.index(p)]) for p in sel})
        _apply_override(rec, override)
        for p in rec.selected:
            self.x[p] = rec.chosen_tokens[p]
            self.decoded[p] = True
        self._apply_eos(rec.selected)
        self.t += 1
        if not keep_logits:
            rec.logits = None
        return rec


def generate_windowed(model, prompt, gen_len, win, override=None, keep_logits=False,
                      eos_id=None, refresh="full"):
    dec = WindowedDecoder(model, prompt, gen_len, win, eos_id=eos_id, refresh=refresh)
    recs = []
    while not dec.done():
        recs.append(dec.step(override, keep_logits))
    return dec.x.copy(), recs


def generate_full(model, prompt, gen_len, k, override=None, keep_logits=False, eos_id=None):
    dec = FullDecoder(model, prompt, gen_len, k, eos_id=eos_id)
    recs = []
    while not dec.done():
        recs.append(dec.step(override, keep_logits))
    return dec.x.copy(), recs


@dataclasses.dataclass(frozen=True)
class PlannedStep:
    refresh: bool
    ctx_len: int
    n_active: int
    n_online: int        # rows computed: ctx_len on a refresh, |A| + |D_p| otherwise
    n_phase_decoded: int
    n_decode: int        # positions decoded by this step


def plan_counts(n_prompt: int, gen_len: int, win: synth.WindowSettings,
                refresh: str = "full") -> List[PlannedStep]:
    """Every count of the schedule without adaptive termination, from counts alone.

    The counts do not depend on which positions get decoded: |A| is
    min(n_active, undecoded left in W_ex), each step decodes min(k, |A|), and
    c = S - u + E (u = undecoded positions at the phase start) or S when
    u < E, because all decoded positions precede the E-th undecoded one.
    """
    S = n_prompt + gen_len
    E, R, k, na = win.external, win.refresh_every, win.unmask_per_step, win.n_active
    u = gen_len
    out: List[PlannedStep] = []
    j = None
    in_window = 0
    dp = prev_dp = 0
    c = 0
    phases = 0
    while u > 0:
        is_refresh = j is None or j >= R or in_window == 0
        if is_refresh:
            c = S - u + E if u >= E else S
            in_window = min(E, u)
            prev_dp, dp = dp, 0
            j = 0
            phases += 1
        n_act = min(na, in_window)
        dec = min(k, n_act)
        if not is_refresh:
            rows = n_act + dp
        elif refresh == "buffer" and phases > 1:
            rows = in_window + prev_dp      # W_ex plus the previous phase's decoded positions
        else:
            rows = c
        out.append(PlannedStep(is_refresh, c, n_act, rows, dp, dec))
        in_window -= dec
        dp += dec
        u -= dec
        j += 1
    return out
