"""Causal assembly of the Phase-1 input (oracle).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.

Eq. 3: Input_0 = [B_0] and, for i > 0, Input_i = [S_sink || Sigma_0 || ... ||
Sigma_{i-1} || B_i], where S_sink is the first s_sink tokens of B_0
(Section 3.1 "Attention sinks"; Algorithm 1) and Sigma_j is the k selected
chunks of block j in positional order.  Every assembled row keeps the global
position of the token it copies (Section 3.1 "Causal Assembly"; Appendix
"RoPE Position ID Assignment", sparse mode), so the assembly is fully
described by the list of global positions, one per row.

The Star Attention baseline prefixes the whole first block instead:
Input_i = [B_0 || B_i] for i > 0 (Section 2 "Background").

The Even-Spaced baseline (Appendix "Even-Spaced") keeps the same sink and
summary slots, but Sigma_j is sigma = k * m single tokens of B_j at evenly
spaced offsets (``scorers.even_spaced_offsets``) rather than k chunks.

Readings taken: a chunk of Sigma_0 that overlaps the sink is kept as a
duplicate row (Eq. 3 taken literally); block 0 gets no sink (Eq. 3).
"""
from __future__ import annotations

import numpy as np

PREFIX_SUMMARY = 0
PREFIX_ANCHOR = 1
PREFIX_EVEN = 2


def phase1_len(L: int, num_blocks: int, block_idx: int, sink: int, chunk: int, topk: int,
               mode: int = PREFIX_SUMMARY) -> int:
    """Number of rows of Input_i, counted from Eq. 3 (summary and Even-Spaced
    modes: one block, one sink, i summaries of k*m rows; anchor mode: two
    blocks)."""
    Lb = L // num_blocks
    if block_idx == 0:
        return Lb
    if mode == PREFIX_ANCHOR:
        return 2 * Lb
    return Lb + sink + block_idx * topk * chunk


def phase1_positions(L: int, num_blocks: int, block_idx: int, sink: int, chunk: int,
                     topk: int, sel_seq=None, mode: int = PREFIX_SUMMARY) -> np.ndarray:
    """Global position of every row of Input_i, built segment by segment in the
    order of Eq. 3.  ``sel_seq [N, k]`` holds the selected chunk indices of
    each block of this sequence (ascending)."""
    Lb = L // num_blocks
    i = block_idx
    segments = []
    if i > 0:
        if mode == PREFIX_ANCHOR:
            segments.append(list(range(0, Lb)))                      # B_0
        elif mode == PREFIX_EVEN:
            from .scorers import even_spaced_offsets
            segments.append(list(range(0, sink)))                    # S_sink
            offs = even_spaced_offsets(Lb, topk * chunk) if topk * chunk else []
            for j in range(i):                                       # Sigma_j
                segments.append([j * Lb + int(o) for o in offs])
        else:
            segments.append(list(range(0, sink)))                    # S_sink
            for j in range(i):                                       # Sigma_j
                if len(sel_seq[j]) != topk:
                    raise ValueError("each block must have exactly topk selected chunks")
                for c in sel_seq[j]:
                    start = j * Lb + int(c) * chunk
                    segments.append(list(range(start, start + chunk)))
    segments.append(list(range(i * Lb, (i + 1) * Lb)))               # B_i
    pos = [p for seg in segments for p in seg]
    return np.array(pos, dtype=np.int64)


def retained_mask(n_rows: int, Lb: int) -> np.ndarray:
    """Rows whose KV is kept after Phase 1: the last |B_i| rows of Input_i
    (Appendix "KV Cache Discard")."""
    keep = np.zeros(n_rows, dtype=bool)
    keep[n_rows - Lb:] = True
    return keep
