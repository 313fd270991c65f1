"""The alternative chunk scorers and the Even-Spaced baseline (oracle).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.

Definitions followed (Appendix "Scoring Heuristic Details"):

* every heuristic scores the non-overlapping contiguous chunks of m tokens of
  a block, keeps the top k and returns them in positional order;
* IDF(t) = log(N / max(df(t), 1)) over the N blocks of the context (Appendix
  "Corpus-Level IDF Table", Eq. idf);
* TF-IDF: the mean of IDF over the chunk's positions (Eq. tfidf);
* BM25: the sum over the chunk's distinct tokens t of
  IDF_BM25(t) * tf(t) (k1 + 1) / (tf(t) + k1 D(C)), with D(C) = 1 - b +
  b |C| / l_bar, k1 = 1.2, b = 0.75, l_bar the mean chunk length of the
  corpus, and IDF_BM25(t) = log((N - df(t) + 0.5) / (df(t) + 0.5) + 1)
  (Eq. bm25);
* Entropy (type-token ratio): distinct tokens of the chunk over its length
  (Eq. entropy);
* Max-IDF: the largest IDF in the chunk (Eq. maxidf);
* Even-Spaced: sigma = k * m token positions of a block, the floors of sigma
  evenly spaced points from 0 to |B| - 1 (Appendix "Even-Spaced").

Precision of the ranking.  The paper computes these scores from an fp32 IDF
table, so a score here is the fp32 number nearest to the exact real value
(ties to even), computed from 50-digit decimal arithmetic and rounded once.
Chunks rank by that fp32 score, higher first, and equal fp32 scores by the
lower chunk index (the tie-break read for Max-IDF).  ``f32_ambiguous`` flags
exact values so close to the midpoint between two fp32 numbers that an
evaluation in fp64 could round them the other way.

Readings taken where the paper is silent or garbled:

* natural logarithm (as for Max-IDF);
* all chunks have m tokens, so l_bar = m and D(C) = 1;
* the Even-Spaced formula names the sink length as the number of points, but
  the text fixes the number of selected tokens at num_chunks * chunk_size:
  sigma = k * m points, the floor taken of the exact quotient
  r (|B| - 1) / (sigma - 1); one point (sigma = 1) is position 0.
"""
from __future__ import annotations

from decimal import Decimal, localcontext

import numpy as np

from . import maxidf

MAXIDF = 0
TFIDF = 1
BM25 = 2
ENTROPY = 3

K1 = Decimal("1.2")
B_BM25 = Decimal("0.75")
_PREC = 50


def _ln(x: Decimal) -> Decimal:
    with localcontext() as ctx:
        ctx.prec = _PREC
        return x.ln()


def to_f32(x: Decimal) -> np.float32:
    """The fp32 number nearest to x, ties to even mantissa (no double
    rounding through fp64)."""
    c = np.float32(float(x))
    cands = [np.nextafter(c, np.float32(-np.inf)), c, np.nextafter(c, np.float32(np.inf))]
    best, best_d = None, None
    for v in cands:
        d = abs(Decimal(float(v)) - x)
        if best is None or d < best_d or (d == best_d and int(v.view(np.uint32)) % 2 == 0):
            best, best_d = v, d
    return np.float32(best)


def f32_ambiguous(x: Decimal, rel: float = 1e-12) -> bool:
    """True when x lies within rel * |x| of the midpoint between its two
    neighbouring fp32 numbers."""
    c = to_f32(x)
    other = np.nextafter(c, np.float32(np.inf) if Decimal(float(c)) < x else np.float32(-np.inf))
    mid = (Decimal(float(c)) + Decimal(float(other))) / 2
    return abs(x - mid) <= Decimal(rel) * abs(x)


def _chunks(ids_seq, num_blocks: int, chunk: int):
    blocks = maxidf.split_blocks(ids_seq, num_blocks)
    Lb = len(blocks[0])
    if Lb % chunk:
        raise ValueError("block length must be a multiple of the chunk size")
    return [[block[c * chunk:(c + 1) * chunk] for c in range(Lb // chunk)] for block in blocks]


def exact_scores(ids_seq, num_blocks: int, chunk: int, vocab: int, scorer: int):
    """Exact score of every chunk of one sequence, as Decimals [N][C]."""
    N = num_blocks
    df = maxidf.document_frequency(ids_seq, num_blocks, vocab)
    lnN = _ln(Decimal(N))
    idf = {}      # df value -> IDF (Eq. idf)
    idf_bm = {}   # df value -> IDF_BM25
    for d in range(0, N + 1):
        idf[d] = lnN - _ln(Decimal(max(d, 1)))
        with localcontext() as ctx:
            ctx.prec = _PREC
            idf_bm[d] = _ln((Decimal(N) - d + Decimal("0.5")) / (Decimal(d) + Decimal("0.5")) + 1)
    out = []
    for block_chunks in _chunks(ids_seq, num_blocks, chunk):
        row = []
        for C in block_chunks:
            with localcontext() as ctx:
                ctx.prec = _PREC
                if scorer == MAXIDF:
                    s = max(idf[int(df[t])] for t in C)
                elif scorer == TFIDF:
                    s = sum((idf[int(df[t])] for t in C), Decimal(0)) / len(C)
                elif scorer == ENTROPY:
                    s = Decimal(len(set(C))) / len(C)
                elif scorer == BM25:
                    l_bar = Decimal(chunk)  # every chunk of the corpus has m tokens
                    D = 1 - B_BM25 + B_BM25 * Decimal(len(C)) / l_bar
                    tf = {}
                    for t in C:
                        tf[t] = tf.get(t, 0) + 1
                    s = sum((idf_bm[int(df[t])] * n * (K1 + 1) / (n + K1 * D)
                             for t, n in tf.items()), Decimal(0))
                else:
                    raise ValueError("unknown scorer")
            row.append(s)
        out.append(row)
    return out


def select_by_score(scores_f32_block, k: int):
    """The k best chunks of one block, best = (fp32 score high, index low),
    returned in ascending (positional) order."""
    C = len(scores_f32_block)
    if not 0 <= k <= C:
        raise ValueError("k must lie in [0, chunks per block]")
    ranked = sorted(range(C), key=lambda c: (-float(scores_f32_block[c]), c))
    return sorted(ranked[:k])


def chunk_summaries(ids, num_blocks: int, chunk: int, topk: int, vocab: int, scorer: int):
    """Summaries of a batch ``ids [batch, L]`` under one scorer.

    Returns (sel [batch, N, k] int64 ascending within a block,
             scores [batch, N, C] fp32 (exact value rounded once),
             ambiguous [batch, N, C] bool (see f32_ambiguous))."""
    ids = np.asarray(ids)
    if ids.ndim == 1:
        ids = ids[None]
    sels, f32s, amb = [], [], []
    for seq in ids:
        ex = exact_scores(seq, num_blocks, chunk, vocab, scorer)
        s32 = np.array([[to_f32(x) for x in row] for row in ex], dtype=np.float32)
        f32s.append(s32)
        amb.append(np.array([[f32_ambiguous(x) for x in row] for row in ex], dtype=bool))
        sels.append([select_by_score(s32[j], topk) for j in range(num_blocks)])
    sel = np.array(sels, dtype=np.int64).reshape(ids.shape[0], num_blocks, topk)
    return sel, np.stack(f32s), np.stack(amb)


def even_spaced_offsets(Lb: int, sigma: int) -> np.ndarray:
    """Offsets within a block of the Even-Spaced summary: floor(r (Lb - 1) /
    (sigma - 1)) for r = 0 .. sigma - 1 (one point: offset 0)."""
    if not 1 <= sigma <= Lb:
        raise ValueError("sigma must lie in [1, Lb]")
    if sigma == 1:
        return np.zeros(1, dtype=np.int64)
    return np.array([(r * (Lb - 1)) // (sigma - 1) for r in range(sigma)], dtype=np.int64)
