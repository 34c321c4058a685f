"""FP8 E4M3 consumer of the per-layer scale (test infrastructure only).

Stage 3 of Algorithm "Geometry-Aware Attention Forward Pass" (Sec. 3.4) up to
the quantised logits, in float64 and in the algorithm's order:
    Q, K = X W^Q, X W^K
    S = Q K^T / sqrt(d_h)                     (per query head h, key head g(h))
    S~ = S / scale
then the OCP E4M3FN code of S~ (``oracle.e4m3.encode``, round to nearest
even, NaN past 464) and the statistics the paper reports: overflow when
|S~| > R_max = 448 (Sec. 1, "Problem formulation"; Table "pretrained":
"Overflow" and "Max Scaled"), and the utilisation max|S~| / 448 (Sec. 1).

Weights are in the PyTorch Linear layout ([n_q d_h, d] rows), so the paper's
W^Q_h is the transpose of rows h d_h .. h d_h + d_h - 1.
"""

from __future__ import annotations

import math

import numpy as np

from . import e4m3


def head_logits(x, wq_rows, wk_rows, h: int, n_kv: int, head_dim: int) -> np.ndarray:
    """S_h = (X W^Q_h)(X W^K_{g(h)})^T / sqrt(d_h) for one query head, float64 [seq, seq]."""
    x = np.asarray(x, dtype=np.float64)
    n_q = np.asarray(wq_rows).shape[0] // head_dim
    g = n_q // n_kv
    j = h // g
    WQh = np.asarray(wq_rows[h * head_dim:(h + 1) * head_dim], dtype=np.float64).T   # d x d_h
    WKj = np.asarray(wk_rows[j * head_dim:(j + 1) * head_dim], dtype=np.float64).T
    Q = x @ WQh
    K = x @ WKj
    return Q @ K.T / math.sqrt(head_dim)


def consume_layer(x, wq_rows, wk_rows, scale: float, n_kv: int, head_dim: int, heads=None,
                  want_codes: bool = True) -> dict:
    """All (or the listed) query heads of one layer: scaled logits S~, their
    E4M3 codes, max |S~| and the overflow count per head."""
    n_q = np.asarray(wq_rows).shape[0] // head_dim
    heads = range(n_q) if heads is None else heads
    out = {"scaled": {}, "codes": {}, "max_abs": {}, "n_over": {}}
    for h in heads:
        s = head_logits(x, wq_rows, wk_rows, h, n_kv, head_dim) / scale
        out["scaled"][h] = s
        if want_codes:
            out["codes"][h] = e4m3.encode(s)
        out["max_abs"][h] = float(np.max(np.abs(s)))
        out["n_over"][h] = int(np.count_nonzero(e4m3.overflows(s)))
    return out


def utilization(max_abs_scaled: float, r_max: float = e4m3.R_MAX) -> float:
    """max|S~| / R_max, the fraction of the E4M3 range the largest logit uses."""
    return max_abs_scaled / r_max
