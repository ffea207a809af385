"""Confidence-based choice of the update set.

Each diffusion step updates the positions the model is most confident about
(Sec. 3.1, update set U(t); Observation 1 ranks undecoded positions by
prediction confidence).  The paper does not define confidence further; the
reading here is greedy decoding:

* the candidate token of a position is the argmax of its logits with the
  [MASK] id excluded (ties go to the lowest token id);
* its confidence is that token's softmax probability, 1 / sum_v exp(l_v - l_max);
* the k positions with the highest confidence are updated (ties go to the
  lowest position); fewer if fewer candidates exist.

The integer decisions (argmax and ranking) are taken on float32 values, the
precision the paper's experiments ran in; confidences are computed in float64
and rounded to float32 before they are compared.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np


def confidence(logits: np.ndarray, mask_id: int) -> Tuple[np.ndarray, np.ndarray]:
    """logits [n, V] -> (token [n] int64, conf [n] float32)."""
    l = np.array(logits, dtype=np.float64, copy=True)
    l[:, mask_id] = -np.inf
    tok = np.argmax(l.astype(np.float32), axis=1)             # first max = lowest id
    lmax = l[np.arange(l.shape[0]), tok]
    conf = 1.0 / np.sum(np.exp(l - lmax[:, None]), axis=1)
    return tok.astype(np.int64), conf.astype(np.float32)


def top1_margin(logits: np.ndarray, mask_id: int) -> np.ndarray:
    """Gap between the best and second-best logit of each row, [MASK] excluded."""
    l = np.array(logits, dtype=np.float64, copy=True)
    l[:, mask_id] = -np.inf
    part = np.sort(l, axis=1)
    return part[:, -1] - part[:, -2]


def select_updates(positions: Sequence[int], conf: Sequence[float], k: int) -> List[int]:
    """The min(k, n) positions with the highest confidence (float32), ties to the
    lowest position; returned in that rank order."""
    c = np.asarray(conf, dtype=np.float32)
    order = sorted(range(len(positions)), key=lambda i: (-float(c[i]), int(positions[i])))
    return [int(positions[i]) for i in order[:k]]
