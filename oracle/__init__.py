"""CPU oracle for the windowed denoising step of Window-Diffusion
(arXiv 2601.20332).

THIS PACKAGE IS TEST INFRASTRUCTURE.  Only the tests, the smoke check and the
CPU-baseline leg of the benchmark may import it.  The GPU library never calls
it, links it or falls back to it, and it shares no code with the GPU library:
the only thing both sides read is the seeded input generator in ``synth``.

It is a plain, slow, float64 NumPy implementation written from the paper:

* ``numerics``  - the per-layer building blocks (RMSNorm, RoPE, bidirectional
  attention, SwiGLU) and the bf16 rounding points of the bf16 datapath;
* ``model``     - the full-sequence forward of a masked diffusion LM
  (Sec. 3.1) and the row-subset forward over a KV cache (Sec. 4.3);
* ``sampler``   - confidence of a position and the update-set selection
  (Sec. 3.1 and Observation 1);
* ``schedule``  - phases, the external/internal windows, buffer set,
  refresh and normal steps (Secs. 4.1-4.3), and the full-sequence
  decoding it approximates (Sec. 3.1).

Every function is pinned by the ``not gpu`` tests against something other
than itself: a pure-Python loop forward, library routines (torch CPU
operators), closed forms and invariants of the method.  Points where the
paper is silent are read as stated in each function's docstring.
"""
from .numerics import round_bf16  # noqa: F401
from .model import OracleModel  # noqa: F401
from .sampler import confidence, select_updates  # noqa: F401
from .schedule import (WindowedDecoder, FullDecoder, plan_counts,  # noqa: F401
                       generate_windowed, generate_full)
