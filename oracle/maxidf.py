"""Max-IDF summary construction, written out from its definition (oracle).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.

Definitions followed (Section 3.1 "Summary generation"; Appendix "Corpus-Level
IDF Table" and "Max-IDF"):

* the context of length L is split into N contiguous logical blocks B_j of
  L/N tokens (Section 3.1; Algorithm 1 input);
* df(t) is the number of blocks that contain token t;
* IDF(t) = log(N / max(df(t), 1)) with the natural logarithm (Eq. idf);
* a block is cut into non-overlapping contiguous chunks of m tokens, and a
  chunk's score is the largest IDF among its tokens (Eq. 2, Eq. maxidf);
* the k best chunks of each block form its summary, returned in positional
  order (Algorithm 1, summary step; Appendix "Scoring Heuristic Details").

Reading taken where the paper is silent: among equal scores the chunk with
the lower index ranks first.
"""
from __future__ import annotations

import math

import numpy as np


def split_blocks(ids_seq, num_blocks: int):
    """The N logical blocks of one sequence, as Python lists of ints."""
    ids_seq = [int(t) for t in ids_seq]
    L = len(ids_seq)
    if num_blocks <= 0 or L % num_blocks:
        raise ValueError("L must be a positive multiple of num_blocks")
    Lb = L // num_blocks
    return [ids_seq[j * Lb:(j + 1) * Lb] for j in range(num_blocks)]


def document_frequency(ids_seq, num_blocks: int, vocab: int) -> np.ndarray:
    """df[t] = number of blocks containing t, counted with Python sets."""
    df = np.zeros(vocab, dtype=np.int64)
    for block in split_blocks(ids_seq, num_blocks):
        for t in set(block):
            df[t] += 1
    return df


def idf_table(df: np.ndarray, num_blocks: int) -> np.ndarray:
    """IDF(t) = ln(N / max(df(t), 1)) for every vocabulary entry (fp64)."""
    return np.array([math.log(num_blocks / max(int(x), 1)) for x in df], dtype=np.float64)


def chunk_scores(ids_seq, idf: np.ndarray, num_blocks: int, chunk: int) -> np.ndarray:
    """score[j, c] = max over the tokens of chunk c of block j of IDF (fp64)."""
    blocks = split_blocks(ids_seq, num_blocks)
    Lb = len(blocks[0])
    if Lb % chunk:
        raise ValueError("block length must be a multiple of the chunk size")
    C = Lb // chunk
    out = np.empty((num_blocks, C), dtype=np.float64)
    for j, block in enumerate(blocks):
        for c in range(C):
            out[j, c] = max(idf[t] for t in block[c * chunk:(c + 1) * chunk])
    return out


def chunk_min_df(ids_seq, df: np.ndarray, num_blocks: int, chunk: int) -> np.ndarray:
    """mindf[j, c] = smallest df among the tokens of chunk c of block j."""
    blocks = split_blocks(ids_seq, num_blocks)
    Lb = len(blocks[0])
    C = Lb // chunk
    out = np.empty((num_blocks, C), dtype=np.int64)
    for j, block in enumerate(blocks):
        for c in range(C):
            out[j, c] = min(int(df[t]) for t in block[c * chunk:(c + 1) * chunk])
    return out


def select_topk(scores_block, k: int):
    """Indices of the k best chunks of one block, best = (score high, index
    low), returned in ascending (positional) order."""
    C = len(scores_block)
    if not 0 <= k <= C:
        raise ValueError("k must lie in [0, chunks per block]")
    ranked = sorted(range(C), key=lambda c: (-float(scores_block[c]), c))
    return sorted(ranked[:k])


def maxidf_summaries(ids, num_blocks: int, chunk: int, topk: int, vocab: int):
    """Summaries for a batch of sequences ``ids [batch, L]``.

    Returns (sel [batch, N, k] int64 ascending within a block,
             mindf [batch, N, C] int64, idf [batch, V] fp64,
             scores [batch, N, C] fp64)."""
    ids = np.asarray(ids)
    if ids.ndim == 1:
        ids = ids[None]
    sels, mindfs, idfs, scores = [], [], [], []
    for seq in ids:
        df = document_frequency(seq, num_blocks, vocab)
        idf = idf_table(df, num_blocks)
        sc = chunk_scores(seq, idf, num_blocks, chunk)
        sels.append([select_topk(sc[j], topk) for j in range(num_blocks)])
        mindfs.append(chunk_min_df(seq, df, num_blocks, chunk))
        idfs.append(idf)
        scores.append(sc)
    sel = np.array(sels, dtype=np.int64).reshape(ids.shape[0], num_blocks, topk)
    return sel, np.stack(mindfs), np.stack(idfs), np.stack(scores)
