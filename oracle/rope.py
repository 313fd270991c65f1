"""Rotary position embedding at preserved global positions (oracle).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.

Appendix "RoPE Position ID Assignment", sparse mode (the mode of every
experiment in the paper): each token of an assembled Phase-1 input keeps the
position id it has in the full context, so a query or key row is rotated by
its own global position whichever block's input it appears in, and the
assembled sequence has gaps where unselected tokens were dropped.

Rotary embedding in the rotate-half form of the model families the paper
evaluates (Qwen3, Llama-3.1): a head vector x of even width d is split into
halves, and pair i < d/2, (x_i, x_{i+d/2}), is turned by the angle p * w_i,

    y_i       = x_i cos(p w_i) - x_{i+d/2} sin(p w_i)
    y_{i+d/2} = x_{i+d/2} cos(p w_i) + x_i sin(p w_i),

with w_i = base^(-2i/d) unless a frequency table is given (a model's scaled
table, e.g. Llama-3.1's, is passed as that table).

Readings: the paper names neither the rotary form nor its base; the
rotate-half form and a caller-given base or table follow the evaluated
models.  Everything is fp64 on inputs already rounded to bf16.
"""
from __future__ import annotations

import numpy as np


def inv_freq(d: int, base: float) -> np.ndarray:
    """w_i = base^(-2i/d), i < d/2, in fp64."""
    if d % 2:
        raise ValueError("head width must be even")
    return np.power(float(base), -2.0 * np.arange(d // 2, dtype=np.float64) / d)


def rope(x, pos, freqs) -> np.ndarray:
    """Rotate every head vector of x (..., n, H, d) by its row's position.

    pos has the shape of x's leading (..., n) axes (the rows' positions);
    freqs is the table w (d/2 values).  Returns fp64 of x's shape."""
    x = np.asarray(x, dtype=np.float64)
    pos = np.asarray(pos, dtype=np.float64)
    w = np.asarray(freqs, dtype=np.float64)
    d = x.shape[-1]
    if d % 2 or w.shape != (d // 2,):
        raise ValueError("need an even head width and d/2 frequencies")
    if pos.shape != x.shape[:-2]:
        raise ValueError("one position per row")
    ang = pos[..., None, None] * w  # (..., n, 1, d/2), broadcast over heads
    c, s = np.cos(ang), np.sin(ang)
    lo, hi = x[..., : d // 2], x[..., d // 2:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)
