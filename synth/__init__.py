"""Seeded synthetic inputs for the windowed denoising step of a masked
diffusion language model: model shapes, window settings, random-init weights
and random prompts.

This module holds none of the method's arithmetic.  It only draws numbers
and stores them (fp32 arrays, or bfloat16 bit patterns obtained by the
standard round-to-nearest-even storage conversion).  Both the CPU oracle and
the GPU path read what it produces; neither one's code lives here.

Workload recipe (the paper evaluates trained LLaDA-8B / Dream-7B checkpoints
on GSM8K, MATH, HumanEval and MBPP; none of that is available, so these
seeded inputs stand in for it, with the models' shapes, the paper's
generation lengths of 256-1024 tokens (Sec. 5.1, Tables 4 and 5) and its
window settings scaled to those lengths):

* every weight matrix and bias is drawn i.i.d. N(0, 0.02) in fp32 and, for
  bf16 models, stored as bf16 (round to nearest even); RMSNorm gains are 1;
* tensor i (in ``tensor_specs`` order) uses its own stream
  ``PCG64(SeedSequence(seed_w).spawn(n_tensors)[i])``;
* prompt ids are uniform on ``[0, vocab) minus {mask_id}``
  (``mask_id = vocab - 1``), drawn from ``seed_p``;
* the batched workload draws prompt lengths uniformly from the integers in
  ``[64, 512]`` with ``seed_l``.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
from typing import Iterator, List, Optional, Sequence, Tuple

import numpy as np

SEED_W = 0
SEED_P = 1
SEED_L = 2

DTYPE_F32 = "f32"
DTYPE_BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class ModelShape:
    """Architecture constants of a LLaDA / Qwen2-style bidirectional decoder."""

    n_layers: int
    hidden: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int
    vocab: int
    dtype: str = DTYPE_BF16
    qkv_bias: bool = False
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0

    @property
    def mask_id(self) -> int:
        return self.vocab - 1

    @property
    def q_dim(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


@dataclasses.dataclass(frozen=True)
class WindowSettings:
    """Dual-window and refresh settings: internal window (active) size, buffer
    size (external window = active + buffer), refresh period in steps and
    tokens unmasked per step."""

    n_active: int
    n_buffer: int
    refresh_every: int
    unmask_per_step: int

    @property
    def external(self) -> int:
        return self.n_active + self.n_buffer


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    window: WindowSettings
    batch: int
    prompt_len: int            # fixed length, or the upper bound when ragged
    gen_len: int
    ragged_prompt: Optional[Tuple[int, int]] = None   # inclusive length range


TINY = ModelShape(n_layers=2, hidden=256, n_heads=4, n_kv_heads=4, head_dim=64,
                  ffn=1024, vocab=1024, dtype=DTYPE_F32, rms_eps=1e-5,
                  rope_theta=10000.0)
LLADA_8B = ModelShape(n_layers=32, hidden=4096, n_heads=32, n_kv_heads=32,
                      head_dim=128, ffn=12288, vocab=126464, dtype=DTYPE_BF16,
                      rms_eps=1e-5, rope_theta=500000.0)
DREAM_7B = ModelShape(n_layers=28, hidden=3584, n_heads=28, n_kv_heads=4,
                      head_dim=128, ffn=18944, vocab=152064, dtype=DTYPE_BF16,
                      qkv_bias=True, rms_eps=1e-6, rope_theta=1000000.0)

WORKLOADS = {
    "tiny": Workload("tiny", TINY, WindowSettings(8, 16, 4, 2), 1, 32, 64),
    "llada8b": Workload("llada8b", LLADA_8B, WindowSettings(32, 64, 8, 1), 1, 128, 256),
    "dream7b": Workload("dream7b", DREAM_7B, WindowSettings(32, 128, 8, 2), 1, 256, 512),
    "llada8b_long": Workload("llada8b_long", LLADA_8B, WindowSettings(64, 256, 16, 2),
                             1, 512, 1024),
    "llada8b_batch16": Workload("llada8b_batch16", LLADA_8B, WindowSettings(32, 128, 8, 1),
                                16, 512, 512, ragged_prompt=(64, 512)),
}


def with_layers(shape: ModelShape, n_layers: int) -> ModelShape:
    """The same per-layer shapes with a different depth."""
    return dataclasses.replace(shape, n_layers=n_layers)


# --------------------------------------------------------------------------
# tensor inventory
# --------------------------------------------------------------------------

def tensor_specs(m: ModelShape) -> List[Tuple[str, Tuple[int, ...], str]]:
    """(name, shape, init) for every weight, in the fixed order the library's
    init call expects.  Linear weights are [out_features, in_features]."""
    specs = [("emb", (m.vocab, m.hidden), "normal")]
    for l in range(m.n_layers):
        p = f"layers.{l}."
        specs.append((p + "attn_norm", (m.hidden,), "ones"))
        specs.append((p + "wq", (m.q_dim, m.hidden), "normal"))
        specs.append((p + "wk", (m.kv_dim, m.hidden), "normal"))
        specs.append((p + "wv", (m.kv_dim, m.hidden), "normal"))
        if m.qkv_bias:
            specs.append((p + "bq", (m.q_dim,), "normal"))
            specs.append((p + "bk", (m.kv_dim,), "normal"))
            specs.append((p + "bv", (m.kv_dim,), "normal"))
        specs.append((p + "wo", (m.hidden, m.q_dim), "normal"))
        specs.append((p + "ffn_norm", (m.hidden,), "ones"))
        specs.append((p + "wg", (m.ffn, m.hidden), "normal"))
        specs.append((p + "wu", (m.ffn, m.hidden), "normal"))
        specs.append((p + "wd", (m.hidden, m.ffn), "normal"))
    specs.append(("final_norm", (m.hidden,), "ones"))
    specs.append(("lm_head", (m.vocab, m.hidden), "normal"))
    return specs


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Storage conversion fp32 -> bf16 bit pattern, round to nearest even
    (finite inputs only)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Storage conversion bf16 bit pattern -> fp32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


class Weights:
    """Deterministic, lazily generated weights of one model.

    ``raw(i)`` is tensor i in its storage form: float32 for fp32 models,
    uint16 bf16 bit patterns for bf16 models.  ``f32(name)`` is the same
    values widened to float32.  Any tensor can be regenerated on its own,
    so an 8B-parameter model never has to sit in host memory whole.
    """

    def __init__(self, shape: ModelShape, seed: int = SEED_W, std: float = 0.02):
        self.shape = shape
        self.specs = tensor_specs(shape)
        self.index = {name: i for i, (name, _, _) in enumerate(self.specs)}
        self.std = std
        self._children = np.random.SeedSequence(seed).spawn(len(self.specs))

    def __len__(self) -> int:
        return len(self.specs)

    def raw(self, i: int) -> np.ndarray:
        name, shp, init = self.specs[i]
        if init == "ones":
            v = np.ones(shp, dtype=np.float32)
        else:
            rng = np.random.Generator(np.random.PCG64(self._children[i]))
            v = rng.standard_normal(shp, dtype=np.float32)
            v *= np.float32(self.std)
        if self.shape.dtype == DTYPE_BF16:
            return f32_to_bf16_bits(v)
        return v

    def f32(self, name: str) -> np.ndarray:
        r = self.raw(self.index[name])
        return bf16_bits_to_f32(r) if r.dtype == np.uint16 else r

    def iter_raw(self, workers: int = 1) -> Iterator[Tuple[int, np.ndarray]]:
        """Yield (i, raw tensor) in order; ``workers`` > 1 draws ahead on threads
        (numpy's generators release the GIL for bulk fills)."""
        if workers <= 1:
            for i in range(len(self.specs)):
                yield i, self.raw(i)
            return
        with _cf.ThreadPoolExecutor(max_workers=workers) as ex:
            futs = {}
            nxt = 0
            for i in range(len(self.specs)):
                while nxt < len(self.specs) and nxt < i + workers:
                    futs[nxt] = ex.submit(self.raw, nxt)
                    nxt += 1
                yield i, futs.pop(i).result()


def prompt_lengths(w: Workload, seed: int = SEED_L) -> List[int]:
    if w.ragged_prompt is None:
        return [w.prompt_len] * w.batch
    lo, hi = w.ragged_prompt
    rng = np.random.Generator(np.random.PCG64(seed))
    return [int(v) for v in rng.integers(lo, hi + 1, size=w.batch)]


def prompts(shape: ModelShape, lengths: Sequence[int], seed: int = SEED_P) -> List[np.ndarray]:
    """One int32 id array per sequence, uniform on [0, vocab) minus {mask_id}.
    With mask_id = vocab - 1 that is uniform on [0, vocab - 1)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    for n in lengths:
        ids = rng.integers(0, shape.vocab - 1, size=int(n)).astype(np.int32)
        out.append(ids)
    return out
