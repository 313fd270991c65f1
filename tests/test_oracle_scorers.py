"""Pins of oracle.scorers (TF-IDF, BM25, Entropy, Even-Spaced; Appendix
"Scoring Heuristic Details").

Each test ties the oracle to something other than its own formula: the
correct fp32 rounding of hand-chosen values (including one that rounding
through fp64 gets wrong), closed forms of special chunks, a hand-worked BM25
chunk, the paper's own statements (TF-IDF equals the mean TF-IDF over types;
Entropy equals a bincount), the exact integer ranking TF-IDF reduces to,
brute-force top-k on tiny blocks, and numpy's linspace.
"""
import itertools
import math
from decimal import Decimal
from fractions import Fraction

import numpy as np
import pytest

from oracle import assembly, maxidf, scorers
from paper_2607_20457_amd import workload


# ------------------------------------------------------------ fp32 rounding --

def test_to_f32_rounds_once_to_nearest_even():
    one = Decimal(1)
    assert scorers.to_f32(one) == np.float32(1.0)
    # the midpoint between 1 and 1 + 2^-23 goes to the even neighbour, 1
    assert scorers.to_f32(one + Decimal(2) ** -24) == np.float32(1.0)
    # the midpoint above 1 + 2^-23 goes to 1 + 2^-22
    assert scorers.to_f32(one + 3 * Decimal(2) ** -24) == np.float32(1 + 2.0 ** -22)
    # just above the first midpoint: 1 + 2^-23.  Through fp64 the 2^-60 is
    # lost and the tie rounds down, which is the double rounding avoided here.
    x = one + Decimal(2) ** -24 + Decimal(2) ** -60
    assert np.float32(float(x)) == np.float32(1.0)
    assert scorers.to_f32(x) == np.float32(1 + 2.0 ** -23)
    assert scorers.f32_ambiguous(x) and scorers.f32_ambiguous(one + Decimal(2) ** -24)
    assert not scorers.f32_ambiguous(Decimal("0.1"))


# ------------------------------------------------------------------ TF-IDF --

def _seq_with_blocks(blocks):
    return np.concatenate([np.asarray(b) for b in blocks])


def test_tfidf_closed_forms():
    # N = 4 blocks of 8 (chunks of 4): chunk 0 of block 0 holds ids that
    # appear nowhere else (score ln 4); chunk 1 of block 0 holds ids present
    # in every block (score 0)
    common = [1, 2, 3, 4]
    blocks = [[10, 11, 12, 13] + common, [20, 21, 22, 23] + common,
              [30, 31, 32, 33] + common, [40, 41, 42, 43] + common]
    ex = scorers.exact_scores(_seq_with_blocks(blocks), 4, 4, 64, scorers.TFIDF)
    assert abs(float(ex[0][0]) - math.log(4)) < 1e-15
    assert ex[0][1] == 0


@pytest.mark.parametrize("seed", range(3))
def test_tfidf_equals_mean_tfidf_over_types(seed):
    # the paper's remark: the positional mean equals sum_t tf(t) idf(t) / |C|
    ids = workload.zipf_ids(50 + seed, 2048, 300)
    N, m = 8, 16
    df = maxidf.document_frequency(ids, N, 300)
    ex = scorers.exact_scores(ids, N, m, 300, scorers.TFIDF)
    for j in range(N):
        for c in range(256 // m):
            C = ids[j * 256 + c * m: j * 256 + (c + 1) * m].tolist()
            types = {t: C.count(t) for t in set(C)}
            ref = sum(n * math.log(N / max(df[t], 1)) for t, n in types.items()) / m
            assert abs(float(ex[j][c]) - ref) < 1e-12


@pytest.mark.parametrize("seed", range(3))
def test_tfidf_ranking_is_the_df_product_ranking(seed):
    # mean of log(N/df) over m positions is decreasing in prod(df): the exact
    # ranking is an integer comparison of products
    ids = workload.zipf_ids(70 + seed, 4096, 200)
    N, m = 8, 16
    df = maxidf.document_frequency(ids, N, 200)
    ex = scorers.exact_scores(ids, N, m, 200, scorers.TFIDF)
    for j in range(N):
        prods = [math.prod(int(df[t]) for t in ids[j * 512 + c * m: j * 512 + (c + 1) * m])
                 for c in range(512 // m)]
        by_score = sorted(range(len(prods)), key=lambda c: (-ex[j][c], c))
        by_prod = sorted(range(len(prods)), key=lambda c: (prods[c], c))
        assert by_score == by_prod


# -------------------------------------------------------------------- BM25 --

def test_bm25_idf_form():
    # log((N - df + 0.5)/(df + 0.5) + 1) is log((N + 1)/(df + 0.5))
    for N in (1, 4, 16, 255):
        for d in range(0, N + 1):
            a = math.log((N - d + 0.5) / (d + 0.5) + 1)
            assert abs(a - math.log((N + 1) / (d + 0.5))) < 1e-14


def test_bm25_hand_worked_chunk():
    # N = 4, m = 4, chunk [x, x, y, z] with df(x) = 1, df(y) = 2, df(z) = 4.
    # D = 1 (every chunk has m tokens); tf weight 2 * 2.2 / (2 + 1.2) = 1.375
    # for x and 2.2 / 2.2 = 1 for y and z.
    x, y, z, f = 7, 8, 9, 5
    blocks = [[x, x, y, z], [y, f, f, z], [f, f, f, z], [f, f, f, z]]
    ex = scorers.exact_scores(_seq_with_blocks(blocks), 4, 4, 16, scorers.BM25)
    want = 1.375 * math.log(5 / 1.5) + math.log(5 / 2.5) + math.log(5 / 4.5)
    assert abs(float(ex[0][0]) - want) < 1e-14


def test_bm25_special_chunks():
    # all-distinct chunk: the tf weight is 1, so the score is the sum of
    # IDF_BM25; one token repeated m times: IDF_BM25 * 2.2 m / (m + 1.2)
    m, N = 8, 2
    blocks = [list(range(100, 108)) + [1] * 8, list(range(200, 208)) + [2] * 8]
    ex = scorers.exact_scores(_seq_with_blocks(blocks), N, m, 256, scorers.BM25)
    assert abs(float(ex[0][0]) - 8 * math.log(3 / 1.5)) < 1e-13
    assert abs(float(ex[0][1]) - math.log(3 / 1.5) * 2.2 * 8 / 9.2) < 1e-13


# ----------------------------------------------------------------- Entropy --

@pytest.mark.parametrize("seed", range(3))
def test_entropy_is_the_bincount_ratio(seed):
    ids = workload.zipf_ids(90 + seed, 2048, 150)
    ex = scorers.exact_scores(ids, 4, 32, 150, scorers.ENTROPY)
    for j in range(4):
        for c in range(16):
            C = ids[j * 512 + c * 32: j * 512 + (c + 1) * 32]
            assert ex[j][c] == Decimal(int((np.bincount(C) > 0).sum())) / 32


def test_entropy_extremes():
    blocks = [[5] * 16 + list(range(16))]
    ex = scorers.exact_scores(_seq_with_blocks(blocks), 1, 16, 64, scorers.ENTROPY)
    assert ex[0] == [Decimal(1) / 16, Decimal(1)]


# ----------------------------------------------------------- top-k, Max-IDF --

@pytest.mark.parametrize("scorer", [scorers.TFIDF, scorers.BM25, scorers.ENTROPY])
@pytest.mark.parametrize("seed", range(4))
def test_topk_unique_by_brute_force(scorer, seed):
    # tiny blocks of <= 8 chunks: exactly one k-subset has every selected
    # chunk ahead of every unselected one on (fp32 score desc, index asc)
    ids = workload.zipf_ids(300 + seed, 3 * 64, 40)
    N, m, k = 3, 8, 3
    sel, s32, _ = scorers.chunk_summaries(ids[None], N, m, k, 40, scorer)
    for j in range(N):
        s = s32[0, j]
        ok = [S for S in itertools.combinations(range(8), k)
              if all((-s[a], a) < (-s[b], b) for a in S for b in set(range(8)) - set(S))]
        assert len(ok) == 1 and list(ok[0]) == sel[0, j].tolist()


def test_maxidf_scorer_matches_the_maxidf_oracle():
    ids = workload.zipf_ids(11, 8192, 2000)
    sel_a, _, _, sc = maxidf.maxidf_summaries(ids[None], 8, 32, 5, 2000)
    sel_b, s32, _ = scorers.chunk_summaries(ids[None], 8, 32, 5, 2000, scorers.MAXIDF)
    assert np.array_equal(sel_a, sel_b)
    assert np.array_equal(s32, sc.astype(np.float32))


# ------------------------------------------------------------- Even-Spaced --

@pytest.mark.parametrize("Lb,sigma", [(8192, 1024), (8192, 512), (4096, 64), (1024, 1000),
                                      (1000, 7), (64, 64), (10, 2)])
def test_even_spaced_matches_linspace(Lb, sigma):
    offs = scorers.even_spaced_offsets(Lb, sigma)
    ref = np.floor(np.linspace(0, Lb - 1, sigma))
    exact = [Fraction(r * (Lb - 1), sigma - 1) for r in range(sigma)]
    for r in range(sigma):
        # numpy's floating point may fall just below an exact integer point
        if exact[r].denominator != 1:
            assert offs[r] == ref[r]
        assert offs[r] == math.floor(exact[r])
    assert offs[0] == 0 and offs[-1] == Lb - 1 and len(offs) == sigma
    gaps = np.diff(offs)
    assert gaps.min() >= 1 and gaps.max() - gaps.min() <= 1


def test_even_spaced_one_point():
    assert scorers.even_spaced_offsets(100, 1).tolist() == [0]


def test_even_spaced_assembly():
    L, N, s, m, k = 4096, 4, 64, 16, 4
    for i in range(N):
        pos = assembly.phase1_positions(L, N, i, s, m, k, None, assembly.PREFIX_EVEN)
        assert len(pos) == assembly.phase1_len(L, N, i, s, m, k, assembly.PREFIX_EVEN)
        assert np.array_equal(pos[-1024:], np.arange(i * 1024, (i + 1) * 1024))
        if i:
            assert np.array_equal(pos[:s], np.arange(s))
            offs = scorers.even_spaced_offsets(1024, k * m)
            for j in range(i):
                seg = pos[s + j * k * m: s + (j + 1) * k * m]
                assert np.array_equal(seg, j * 1024 + offs)
