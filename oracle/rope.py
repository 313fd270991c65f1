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

The same appendix describes a contiguous mode (unused in the paper's
experiments): block i's assembled input is renumbered 0 .. n_i - 1 for its
Phase-1 pass, and the Phase-2 query positions start just past the longest
assembled Phase-1 input.  In sparse mode a query keeps its place after the
whole context.

Readings: the paper names neither the rotary form nor its base; the
rotate-half form and a caller-given base or table follow the evaluated
models.  "Just past the longest assembled Phase-1 length" is read as: the
first query (or generated) token after the context has position
max_i n_i, the next one max_i n_i + 1, and so on.  Everything is fp64 on
inputs already rounded to bf16.
"""
from __future__ import annotations

import numpy as np

from . import assembly

SPARSE = 0
CONTIGUOUS = 1


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


def phase1_rope_positions(L: int, num_blocks: int, block_idx: int, sink: int, chunk: int,
                          topk: int, sel_seq=None, prefix_mode: int = assembly.PREFIX_SUMMARY,
                          pos_mode: int = SPARSE) -> np.ndarray:
    """Rotary position of every row of block i's assembled Phase-1 input:
    its global position (sparse) or its row index (contiguous)."""
    if pos_mode == SPARSE:
        return assembly.phase1_positions(L, num_blocks, block_idx, sink, chunk, topk, sel_seq,
                                         prefix_mode)
    n = assembly.phase1_len(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode)
    return np.arange(n, dtype=np.int64)


def query_positions(L: int, num_blocks: int, sink: int, chunk: int, topk: int, Tq: int,
                    G: int = 0, prefix_mode: int = assembly.PREFIX_SUMMARY,
                    pos_mode: int = SPARSE) -> np.ndarray:
    """Rotary positions of Tq Phase-2 tokens that follow G earlier query or
    generated tokens: after the context (sparse), or after the longest
    assembled Phase-1 input (contiguous)."""
    if pos_mode == SPARSE:
        first = L
    else:
        first = max(assembly.phase1_len(L, num_blocks, i, sink, chunk, topk, prefix_mode)
                    for i in range(num_blocks))
    return first + G + np.arange(Tq, dtype=np.int64)


def assembled_rope(x, src_pos, rot_pos, freqs) -> np.ndarray:
    """Rows of a per-position tensor x [L, H, d] at the global positions
    src_pos, each rotated by its entry of rot_pos (fp64)."""
    rows = np.asarray(x, dtype=np.float64)[np.asarray(src_pos, dtype=np.int64)]
    return rope(rows, np.asarray(rot_pos), freqs)
