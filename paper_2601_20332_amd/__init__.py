"""Python binding of libwd, the MI355X windowed-denoising library (include/wd.h).

Argument marshalling only: every step of the method runs in libwd's HIP
kernels.  PyTorch supplies device memory (the packed-weight buffer and the
generation workspace are torch uint8 tensors) and the HIP stream.  Importing
this package fails loudly when libwd.so has not been built.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwd.so")

WD_OK = 0
WD_ERR_INVALID_ARG = -1
WD_ERR_OUT_OF_MEMORY = -2
WD_ERR_DEVICE = -3
WD_ERR_STATE = -4
WD_ERR_UNSUPPORTED = -5
WD_DTYPE_F32 = 0
WD_DTYPE_BF16 = 1

EXPORTED = ["wd_weight_count", "wd_weight_shape", "wd_model_bytes", "wd_init_model",
            "wd_free_model", "wd_seq_bytes", "wd_prefill_prompt", "wd_slide_window",
            "wd_refresh_buffer", "wd_step", "wd_full_step", "wd_get_state", "wd_debug_logits",
            "wd_debug_kv", "wd_free_seq", "wd_plan", "wd_last_error", "wd_profile_enable",
            "wd_profile_read", "wd_seq_ends", "wd_debug_weight_row", "wd_debug_keep_logits", "wd_measure_peaks",
            "wd_debug_gemm_plan", "wd_step_noalloc"]


class WdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"wd status {status}: {msg}")
        self.status = status


class ModelConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("mask_id", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("qkv_bias", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("weight_fp8", ctypes.c_int32)]


class WindowConfig(ctypes.Structure):
    _fields_ = [("n_active", ctypes.c_int32), ("n_buffer", ctypes.c_int32),
                ("refresh_every", ctypes.c_int32), ("unmask_per_step", ctypes.c_int32),
                ("stop_at_eos", ctypes.c_int32), ("eos_id", ctypes.c_int32),
                ("buffer_refresh", ctypes.c_int32)]


class StepOut(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int32), ("is_refresh", ctypes.c_int32),
                ("n_rows", ctypes.c_int32), ("n_selected", ctypes.c_int32),
                ("positions", ctypes.POINTER(ctypes.c_int32)),
                ("tokens", ctypes.POINTER(ctypes.c_int32)),
                ("conf", ctypes.POINTER(ctypes.c_float))]


def _load() -> ctypes.CDLL:
    # PyTorch ships its own HIP runtime (same soname as /opt/rocm's).  Loading
    # torch first makes libwd bind to that one, so a process never holds two
    # HIP/HSA runtimes, whatever order the caller imports things in.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2601_20332_amd/build.py` "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.c_void_p
    i32, sz = ctypes.c_int32, ctypes.c_size_t
    pi32 = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "wd_weight_count": (i32, [ctypes.POINTER(ModelConfig)]),
        "wd_weight_shape": (i32, [ctypes.POINTER(ModelConfig), i32, ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64)]),
        "wd_model_bytes": (sz, [ctypes.POINTER(ModelConfig)]),
        "wd_init_model": (i32, [ctypes.POINTER(ModelConfig), ctypes.POINTER(P), i32, P, sz, P,
                                ctypes.POINTER(P)]),
        "wd_free_model": (None, [P]),
        "wd_seq_bytes": (sz, [P, ctypes.POINTER(WindowConfig), i32, pi32, i32]),
        "wd_prefill_prompt": (i32, [P, pi32, pi32, i32, i32, ctypes.POINTER(WindowConfig), P, sz,
                                    ctypes.POINTER(P)]),
        "wd_slide_window": (i32, [P]),
        "wd_refresh_buffer": (i32, [P]),
        "wd_step": (i32, [P, ctypes.POINTER(StepOut)]),
        "wd_step_noalloc": (i32, [P, ctypes.POINTER(StepOut)]),
        "wd_full_step": (i32, [P, ctypes.POINTER(StepOut)]),
        "wd_get_state": (i32, [P, pi32, ctypes.POINTER(ctypes.c_uint8), pi32]),
        "wd_seq_ends": (i32, [P, pi32]),
        "wd_debug_weight_row": (i32, [P, i32, i32, ctypes.POINTER(ctypes.c_float),
                                      ctypes.POINTER(ctypes.c_float)]),
        "wd_debug_keep_logits": (i32, [P, i32]),
        "wd_debug_logits": (i32, [P, ctypes.POINTER(ctypes.c_float), pi32, i32, pi32]),
        "wd_debug_kv": (i32, [P, i32, i32, ctypes.POINTER(ctypes.c_float),
                              ctypes.POINTER(ctypes.c_float), i32, pi32]),
        "wd_free_seq": (None, [P]),
        "wd_plan": (i32, [i32, i32, ctypes.POINTER(WindowConfig), i32, pi32, pi32, pi32, pi32, pi32]),
        "wd_debug_gemm_plan": (i32, [i32, i32, i32, i32, i32, pi32]),
        "wd_last_error": (ctypes.c_char_p, []),
        "wd_profile_enable": (i32, [P, i32]),
        "wd_measure_peaks": (i32, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
        "wd_profile_read": (i32, [P, i32, ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_double),
                                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


lib = _load()


def _check(status: int) -> None:
    if status != WD_OK:
        raise WdError(status, lib.wd_last_error().decode())


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _f32p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))


def model_config(*, n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab, mask_id, dtype,
                 qkv_bias, rms_eps, rope_theta, weight_fp8: bool = False) -> ModelConfig:
    """weight_fp8 selects the FP8-weight variant (bf16 models; not the paper's precision)."""
    return ModelConfig(n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab, mask_id,
                       WD_DTYPE_BF16 if dtype in ("bf16", WD_DTYPE_BF16) else WD_DTYPE_F32,
                       int(bool(qkv_bias)), rms_eps, rope_theta, int(bool(weight_fp8)))


def window_config(n_active, n_buffer, refresh_every, unmask_per_step,
                  eos_id: Optional[int] = None, buffer_refresh: bool = False) -> WindowConfig:
    """eos_id: None keeps adaptive termination off; a token id turns it on.
    buffer_refresh selects the buffer-only refresh variant (not the paper's)."""
    stop, eos = (0, -1) if eos_id is None else (1, int(eos_id))
    return WindowConfig(n_active, n_buffer, refresh_every, unmask_per_step, stop, eos,
                        int(bool(buffer_refresh)))


# ---- device buffers (torch is plumbing: memory and stream) --------------------------------

def _device_bytes(nbytes: int, device):
    import torch
    t = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-t.data_ptr()) % 256
    return t, t.data_ptr() + off


def _stream_handle(device):
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def wd_weight_count(cfg: ModelConfig) -> int:
    return lib.wd_weight_count(ctypes.byref(cfg))


def wd_weight_shape(cfg: ModelConfig, i: int):
    r, c = ctypes.c_int64(), ctypes.c_int64()
    _check(lib.wd_weight_shape(ctypes.byref(cfg), i, ctypes.byref(r), ctypes.byref(c)))
    return r.value, c.value


def wd_model_bytes(cfg: ModelConfig) -> int:
    return lib.wd_model_bytes(ctypes.byref(cfg))


class Model:
    """A packed model on the GPU: the library handle plus the torch buffer it lives in."""

    def __init__(self, cfg: ModelConfig, handle: ctypes.c_void_p, buf, device):
        self.cfg, self.handle, self._buf, self.device = cfg, handle, buf, device

    def free(self):
        if self.handle:
            lib.wd_free_model(self.handle)
            self.handle = None
            self._buf = None

    def __del__(self):
        self.free()


def wd_init_model(cfg: ModelConfig, weights: Sequence, device="cuda") -> Model:
    """weights: device tensors (fp32, or bf16 bits as int16/uint16/bfloat16) in
    wd_weight_count order."""
    n = len(weights)
    nbytes = wd_model_bytes(cfg)
    if nbytes == 0:
        raise WdError(WD_ERR_UNSUPPORTED, "configuration not supported")
    buf, ptr = _device_bytes(nbytes, device)
    ptrs = (ctypes.c_void_p * n)(*[w.data_ptr() for w in weights])
    h = ctypes.c_void_p()
    _check(lib.wd_init_model(ctypes.byref(cfg), ptrs, n, ctypes.c_void_p(ptr), nbytes,
                             _stream_handle(device), ctypes.byref(h)))
    return Model(cfg, h, buf, device)


@dataclasses.dataclass
class StepResult:
    step: int
    is_refresh: bool
    n_rows: int
    n_selected: int
    positions: np.ndarray   # [batch, k], -1 where unused
    tokens: np.ndarray
    conf: np.ndarray


class Generation:
    """One batch of sequences being decoded (library handle + workspace)."""

    def __init__(self, model: Model, handle, buf, batch, k, lens):
        self.model, self.handle, self._buf = model, handle, buf
        self.batch, self.k, self.lens = batch, k, lens

    def free(self):
        if self.handle:
            lib.wd_free_seq(self.handle)
            self.handle = None
            self._buf = None

    def __del__(self):
        self.free()


def wd_seq_bytes(model: Model, win: WindowConfig, prompt_lens: Sequence[int], gen_len: int) -> int:
    lens = np.ascontiguousarray(prompt_lens, dtype=np.int32)
    return lib.wd_seq_bytes(model.handle, ctypes.byref(win), len(lens), _i32p(lens), gen_len)


def wd_prefill_prompt(model: Model, prompts: Sequence[np.ndarray], gen_len: int,
                      win: WindowConfig) -> Generation:
    lens = np.array([len(p) for p in prompts], dtype=np.int32)
    ids = np.ascontiguousarray(np.concatenate([np.asarray(p, dtype=np.int32) for p in prompts])
                               if len(prompts) else np.zeros(0, np.int32), dtype=np.int32)
    nbytes = wd_seq_bytes(model, win, lens, gen_len)
    if nbytes == 0:
        raise WdError(WD_ERR_INVALID_ARG, "invalid generation arguments")
    buf, ptr = _device_bytes(nbytes, model.device)
    h = ctypes.c_void_p()
    _check(lib.wd_prefill_prompt(model.handle, _i32p(ids), _i32p(lens), len(lens), gen_len,
                                 ctypes.byref(win), ctypes.c_void_p(ptr), nbytes, ctypes.byref(h)))
    return Generation(model, h, buf, len(lens), win.unmask_per_step,
                      [int(v) + gen_len for v in lens])


def _step(fn, gen: Generation, want: bool) -> Optional[StepResult]:
    if not want:
        _check(fn(gen.handle, None))
        return None
    n = gen.batch * gen.k
    pos = np.empty(n, np.int32)
    tok = np.empty(n, np.int32)
    conf = np.empty(n, np.float32)
    out = StepOut(0, 0, 0, 0, _i32p(pos), _i32p(tok), _f32p(conf))
    _check(fn(gen.handle, ctypes.byref(out)))
    return StepResult(out.step, bool(out.is_refresh), out.n_rows, out.n_selected,
                      pos.reshape(gen.batch, gen.k), tok.reshape(gen.batch, gen.k),
                      conf.reshape(gen.batch, gen.k))


def wd_step(gen: Generation, want_result: bool = True) -> Optional[StepResult]:
    return _step(lib.wd_step, gen, want_result)


def wd_step_noalloc(gen: Generation, want_result: bool = True) -> Optional[StepResult]:
    """wd_step with its scratch in the library's static device array (no allocation)."""
    return _step(lib.wd_step_noalloc, gen, want_result)


def wd_full_step(gen: Generation, want_result: bool = True) -> Optional[StepResult]:
    return _step(lib.wd_full_step, gen, want_result)


def wd_slide_window(gen: Generation) -> None:
    _check(lib.wd_slide_window(gen.handle))


def wd_refresh_buffer(gen: Generation) -> None:
    _check(lib.wd_refresh_buffer(gen.handle))


def wd_get_state(gen: Generation):
    total = sum(gen.lens)
    tok = np.empty(total, np.int32)
    dec = np.empty(total, np.uint8)
    t = ctypes.c_int32()
    _check(lib.wd_get_state(gen.handle, _i32p(tok), dec.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                            ctypes.byref(t)))
    out_t, out_d, o = [], [], 0
    for n in gen.lens:
        out_t.append(tok[o:o + n])
        out_d.append(dec[o:o + n].astype(bool))
        o += n
    return out_t, out_d, t.value


def wd_debug_weight_row(model: Model, tensor: int, row: int, in_features: int):
    """(values [in_features] as the GEMMs use them before scaling, fp8 row scale)."""
    vals = np.empty(in_features, np.float32)
    sc = ctypes.c_float()
    _check(lib.wd_debug_weight_row(model.handle, int(tensor), int(row), _f32p(vals), ctypes.byref(sc)))
    return vals, sc.value


def wd_seq_ends(gen: Generation) -> np.ndarray:
    """Live end of each sequence (one past its first decoded <eos>, else its length)."""
    out = np.empty(gen.batch, np.int32)
    _check(lib.wd_seq_ends(gen.handle, _i32p(out)))
    return out


def wd_debug_keep_logits(gen: Generation, on: bool = True) -> None:
    _check(lib.wd_debug_keep_logits(gen.handle, int(bool(on))))


def wd_debug_logits(gen: Generation):
    V = gen.model.cfg.vocab
    n = ctypes.c_int32()
    probe = np.empty(1, np.float32)
    st = lib.wd_debug_logits(gen.handle, _f32p(probe), None, 0, ctypes.byref(n))
    if st not in (WD_OK, WD_ERR_OUT_OF_MEMORY):
        _check(st)
    cap = max(1, n.value)
    logits = np.empty((cap, V), np.float32)
    pos = np.empty(cap, np.int32)
    _check(lib.wd_debug_logits(gen.handle, _f32p(logits), _i32p(pos), cap, ctypes.byref(n)))
    return logits[:n.value], pos[:n.value]


def wd_debug_kv(gen: Generation, layer: int, b: int):
    c = gen.model.cfg
    cap = gen.lens[b]
    k = np.empty((cap, c.n_kv_heads, c.head_dim), np.float32)
    v = np.empty_like(k)
    ctx = ctypes.c_int32()
    _check(lib.wd_debug_kv(gen.handle, layer, b, _f32p(k), _f32p(v), cap, ctypes.byref(ctx)))
    return k[:ctx.value], v[:ctx.value]


def wd_plan(n_prompt: int, gen_len: int, win: WindowConfig):
    n = lib.wd_plan(n_prompt, gen_len, ctypes.byref(win), 0, None, None, None, None, None)
    if n < 0:
        raise WdError(WD_ERR_INVALID_ARG, lib.wd_last_error().decode())
    arrs = {k: np.empty(n, np.int32) for k in ("is_refresh", "ctx_len", "n_active", "n_rows",
                                               "n_decode")}
    lib.wd_plan(n_prompt, gen_len, ctypes.byref(win), n, *[_i32p(arrs[k]) for k in
                                                            ("is_refresh", "ctx_len", "n_active",
                                                             "n_rows", "n_decode")])
    return arrs


GEMM_PLAN_FIELDS = ("kernel", "rows", "features", "splits", "k_steps_per_split", "workgroups",
                    "waves", "accepted")


def wd_debug_gemm_plan(M: int, N: int, K: int, fp8: bool = False, max_splits: int = 1 << 20):
    """The bf16 projection GEMM's launch plan for (M, N, K) (host only)."""
    out = np.zeros(8, np.int32)
    _check(lib.wd_debug_gemm_plan(int(M), int(N), int(K), int(bool(fp8)), int(max_splits),
                                  _i32p(out)))
    return dict(zip(GEMM_PLAN_FIELDS, (int(v) for v in out)))


def wd_profile_enable(model: Model, enable: bool = True) -> None:
    _check(lib.wd_profile_enable(model.handle, int(bool(enable))))


# kernel classes of wd_profile_read
WD_PROF_ALL, WD_PROF_GEMM_ROWS, WD_PROF_GEMM_TILED, WD_PROF_GEMM_F32, WD_PROF_ATTN = 0, 1, 2, 3, 4


def wd_profile_read(model: Model, kernel: int = WD_PROF_ALL):
    """(launches, total_ms, algorithmic bytes, algorithmic flops) of the GEMM
    launches of one kernel class recorded since profiling was enabled."""
    n, ms, by, fl = ctypes.c_int64(), ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib.wd_profile_read(model.handle, int(kernel), ctypes.byref(n), ctypes.byref(ms),
                               ctypes.byref(by), ctypes.byref(fl)))
    return n.value, ms.value, by.value, fl.value


def wd_measure_peaks(model: Model):
    """(dense bf16 MFMA TFLOP/s, HBM read GB/s) measured on the model's GPU."""
    t, g = ctypes.c_double(), ctypes.c_double()
    _check(lib.wd_measure_peaks(model.handle, ctypes.byref(t), ctypes.byref(g)))
    return t.value, g.value


def wd_last_error() -> str:
    return lib.wd_last_error().decode()
