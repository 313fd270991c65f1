"""GPU parity of pulsar_chunk_summaries (TF-IDF, BM25, Entropy, Max-IDF)
with oracle.scorers.

The oracle's score is the exact value rounded once to fp32; the kernel sums
in fp64 and rounds once.  They must agree bit for bit except on chunks whose
exact score lies within 1e-12 (relative) of an fp32 rounding midpoint, where
one ulp either way is allowed.  The selected chunks must be the oracle's;
should an allowed one-ulp difference reorder a block, the selection must
then be the top-k of the kernel's own scores.
"""
import numpy as np
import pytest
import torch

import paper_2607_20457_amd as P
from oracle import scorers
from paper_2607_20457_amd import workload
from tests._helpers import gpu_available, to_dev_i32

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]

SCORERS = [P.SCORE_TFIDF, P.SCORE_BM25, P.SCORE_ENTROPY, P.SCORE_MAXIDF]
NAMES = {P.SCORE_TFIDF: "tfidf", P.SCORE_BM25: "bm25", P.SCORE_ENTROPY: "entropy",
         P.SCORE_MAXIDF: "maxidf"}


def _check(ids, N, m, k, V, scorer):
    """Both paths against the oracle: with the size query's workspace (split
    over blocks and vocabulary where the shapes allow) and without one (one
    workgroup per sequence)."""
    sel_ref, s_ref, amb = scorers.chunk_summaries(ids, N, m, k, V, scorer)
    d_ids = to_dev_i32(ids)
    need = P.chunk_workspace_bytes(ids.shape[0], ids.shape[1], N, m, V, scorer)
    for ws in ("auto", None) if need else (None,):
        print(f"scorer parity: {NAMES[scorer]} batch={ids.shape[0]} L={ids.shape[1]} N={N} m={m} "
              f"k={k} V={V} path={'split' if ws else 'one workgroup per sequence'}", flush=True)
        sel, s = P.chunk_summaries(d_ids, N, m, k, V, scorer, return_scores=True, workspace=ws)
        torch.cuda.synchronize()
        sel, s = sel.cpu().numpy(), s.cpu().numpy()
        exact = ~amb
        assert np.array_equal(s[exact].view(np.uint32), s_ref[exact].view(np.uint32)), \
            f"{NAMES[scorer]}: fp32 scores differ on {(s[exact] != s_ref[exact]).sum()} chunks"
        if amb.any():
            d = np.abs(s[amb].view(np.int32).astype(np.int64) - s_ref[amb].view(np.int32))
            assert d.max() <= 1
        if np.array_equal(s.view(np.uint32), s_ref.view(np.uint32)):
            assert np.array_equal(sel, sel_ref)
        else:
            for bb in range(ids.shape[0]):
                for j in range(N):
                    assert sel[bb, j].tolist() == scorers.select_by_score(s[bb, j], k)
    return sel, s


@pytest.mark.parametrize("scorer", SCORERS)
@pytest.mark.parametrize("name", ["tiny", "llama8b_32k", "llama8b_128k"])
def test_config_workloads(scorer, name):
    cfg = workload.CONFIGS[name]
    ids = workload.make_ids(cfg, batch=1)
    _check(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab, scorer)


@pytest.mark.parametrize("scorer", SCORERS)
@pytest.mark.parametrize("m", [4, 8, 64, 256])
def test_chunk_sizes(scorer, m):
    L, N = 8192, 4
    ids = workload.zipf_ids(600 + m, L, 700)[None]
    C = L // N // m
    for k in sorted({0, 1, C // 3, C}):
        _check(ids, N, m, k, 700, scorer)


@pytest.mark.parametrize("scorer", SCORERS)
def test_discriminative_vocab_batch(scorer):
    ids = np.stack([workload.zipf_ids(1200 + b, 32768, 512) for b in range(3)])
    _check(ids, 8, 32, 16, 512, scorer)


@pytest.mark.parametrize("scorer", SCORERS)
def test_split_path_batch16(scorer):
    # the largest batch the split path takes, 16 blocks (a nibble df table)
    ids = np.stack([workload.zipf_ids(1300 + b, 16384, 3000) for b in range(16)])
    assert P.chunk_workspace_bytes(16, 16384, 16, 16, 3000, scorer) > 0
    _check(ids, 16, 16, 7, 3000, scorer)


@pytest.mark.parametrize("scorer", SCORERS)
def test_degenerate_inputs(scorer):
    # one repeated id: every chunk ties, the first k chunks win
    same = np.full((1, 4096), 3, dtype=np.int32)
    sel, _ = _check(same, 4, 16, 5, 8, scorer)
    assert (sel == np.arange(5)).all()
    # a single block (N = 1: every IDF is 0, BM25's is ln(2/1.5))
    _check(workload.zipf_ids(5, 2048, 90)[None], 1, 16, 7, 90, scorer)
    # a ragged vocabulary size and 16 blocks
    _check(workload.zipf_ids(6, 16 * 256, 33)[None], 16, 32, 3, 33, scorer)


def test_maxidf_scorer_equals_the_maxidf_entry_point():
    cfg = workload.CONFIGS["llama8b_32k"]
    ids = to_dev_i32(workload.make_ids(cfg, batch=2))
    a, mindf = P.maxidf_summaries(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab,
                                  return_mindf=True)
    b, s = P.chunk_summaries(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab,
                             P.SCORE_MAXIDF, return_scores=True)
    assert torch.equal(a, b)
    ref = np.log(cfg.num_blocks / mindf.cpu().numpy().astype(np.float64)).astype(np.float32)
    assert np.array_equal(s.cpu().numpy(), ref)


@pytest.mark.parametrize("scorer", SCORERS)
def test_planted_needles(scorer):
    # 16 planted df = 1 ids on a V = 512 Zipf background (no natural df = 1)
    base = workload.zipf_ids(77, 32768, 512)
    ids, _, pos = workload.plant_needles(78, base, 16, 1024)
    sel, _ = _check(ids[None], 8, 32, 16, 1024, scorer)
    if scorer == P.SCORE_MAXIDF:
        assert all((p % 4096) // 32 in sel[0, p // 4096] for p in pos)


def test_split_path_in_a_graph_replays():
    # As for Max-IDF: captured into a graph, the split scorer path's replays
    # equal the eager result bit for bit, with eager calls between them.
    cfg = workload.CONFIGS["llama8b_32k"]
    N, m, k, V = cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab
    ids = to_dev_i32(workload.make_ids(cfg, batch=2))
    other = to_dev_i32(np.stack([workload.zipf_ids(7100 + b, cfg.L, V) for b in range(2)]))
    need = P.chunk_workspace_bytes(2, cfg.L, N, m, V, P.SCORE_BM25)
    assert need > 0
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    eager = P.chunk_summaries(ids, N, m, k, V, P.SCORE_BM25, return_scores=True, workspace=ws)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        P.chunk_summaries(ids, N, m, k, V, P.SCORE_BM25, return_scores=True, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured = P.chunk_summaries(ids, N, m, k, V, P.SCORE_BM25, return_scores=True,
                                     workspace=ws)
    for rep in range(3):
        print(f"scorer split graph replay {rep}", flush=True)
        for t in captured:
            t.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(captured, eager):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), f"replay {rep}"
        P.chunk_summaries(other, N, m, k, V, P.SCORE_ENTROPY, workspace=ws)
        torch.cuda.synchronize()
