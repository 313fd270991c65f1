"""GPU parity of Max-IDF selection and the Eq. 3 position map against the
fp64 oracle.  Selections, chunk minima and positions must match bit for bit."""
import math

import numpy as np
import pytest
import torch

import paper_2607_20457_amd as P
from oracle import assembly, maxidf
from paper_2607_20457_amd import workload
from tests._helpers import gpu_available, to_dev_i32

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _check(ids, N, m, k, V, idf_too=True, single=True):
    """Both paths against the oracle: with the size query's workspace (split
    over blocks and vocabulary where the shapes allow) and without one (one
    workgroup per sequence).  Their outputs must also agree bit for bit."""
    sel_ref, mindf_ref, idf_ref, _ = maxidf.maxidf_summaries(ids, N, m, k, V)
    d_ids = to_dev_i32(ids)
    need = P.maxidf_workspace_bytes(ids.shape[0], ids.shape[1], N, m, V)
    outs = []
    for ws in (("auto", None) if single else ("auto",)) if need else (None,):
        print(f"maxidf parity: batch={ids.shape[0]} L={ids.shape[1]} N={N} m={m} k={k} V={V} "
              f"path={'split' if ws else 'one workgroup per sequence'}", flush=True)
        if idf_too:
            sel, mindf, idf = P.maxidf_summaries(d_ids, N, m, k, V, return_mindf=True,
                                                 return_idf=True, workspace=ws)
        else:
            (sel, mindf), idf = P.maxidf_summaries(d_ids, N, m, k, V, return_mindf=True,
                                                   workspace=ws), None
        torch.cuda.synchronize()
        assert np.array_equal(mindf.cpu().numpy(), mindf_ref)
        assert np.array_equal(sel.cpu().numpy(), sel_ref)
        if idf_too:
            np.testing.assert_allclose(idf.cpu().numpy(), idf_ref, rtol=2e-6, atol=2e-6)
        outs.append((sel, mindf, idf))
    if len(outs) == 2 and idf_too:
        assert torch.equal(outs[0][2], outs[1][2])       # the same fp32 IDF values
    return outs[-1][0]


@pytest.mark.parametrize("name", ["tiny", "llama8b_32k", "llama8b_128k"])
def test_config_workloads(name):
    cfg = workload.CONFIGS[name]
    ids = workload.make_ids(cfg, batch=1)
    _check(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab)


def test_needles_config_selects_planted_needles_when_discriminative():
    # V=512 background: no natural df=1 ids, so every planted needle chunk wins
    cfg = workload.Config("needles512", L=32768, vocab=512, num_blocks=8, sink=64, chunk=32,
                          topk=16, Hq=1, Hkv=1, d=64)
    base = workload.zipf_ids(77, cfg.L, 512)
    ids, _, pos = workload.plant_needles(78, base, 16, 1024)
    sel = _check(ids[None], 8, 32, 16, 1024)[0].cpu().numpy()
    for p in pos:
        assert (p % cfg.Lb) // 32 in sel[p // cfg.Lb]


@pytest.mark.parametrize("vocab,N,L", [(512, 8, 32768), (2048, 8, 32768), (512, 16, 131072),
                                       (2048, 16, 131072)])
def test_discriminative_vocab(vocab, N, L):
    ids = np.stack([workload.zipf_ids(1000 + vocab + b, L, vocab) for b in range(2)])
    _check(ids, N, 32, 16, vocab)


@pytest.mark.parametrize("m", [4, 8, 16, 64, 128, 256])
def test_chunk_sizes(m):
    L, N = 8192, 4
    ids = workload.zipf_ids(500 + m, L, 700)[None]
    C = L // N // m
    for k in sorted({0, 1, C // 3, C}):
        _check(ids, N, m, k, 700, idf_too=False)


def test_batch8_at_128k():
    cfg = workload.CONFIGS["sweep_128k_b4"]
    ids = workload.make_ids(cfg, batch=8)
    _check(ids, cfg.num_blocks, cfg.chunk, 32, cfg.vocab, idf_too=False)


@pytest.mark.parametrize("L,N,m", [(8192, 1, 32), (16384, 1, 16), (131072, 2, 32),
                                   (131072, 8, 64), (32768, 4, 16)])
def test_resident_block_layouts(L, N, m):
    # The register-resident kernel with one round (8192 ids) per block, where
    # block 0 is also the last block when N = 1, and with several rounds per
    # block, where the first block's rounds test for never-seen ids.
    ids = workload.zipf_ids(5000 + L // 8192 + N, L, 128256)[None]
    print(f"maxidf resident: L={L} N={N} m={m}", flush=True)
    _check(ids, N, m, min(6, L // N // m), 128256)


def test_resident_tiny_vocabularies():
    # every lane stamps the same few bytes: one id (df = N everywhere) and
    # three ids, one of them absent from the last block
    _check(np.zeros((1, 16384), dtype=np.int32), 2, 16, 5, 1)
    ids = (np.arange(32768, dtype=np.int32) % 3)[None]
    ids[0, 24576:] = np.where(ids[0, 24576:] == 2, 0, ids[0, 24576:])
    _check(ids, 4, 32, 3, 3)


def test_single_block_and_adversarial_contention():
    ids = workload.zipf_ids(9, 4096, 3000)[None]
    sel = _check(ids, 1, 16, 7, 3000)
    assert sel.cpu().numpy()[0, 0].tolist() == list(range(7))
    same = np.full((1, 8192), 17, dtype=np.int32)            # every lane hits one LDS word
    _check(same, 8, 32, 5, 64)
    two = (np.arange(16384, dtype=np.int32) % 2)[None] * 1000  # two-token alphabet
    _check(two, 16, 16, 3, 1001)
    ragged_vocab = workload.zipf_ids(10, 6144, 33)[None]      # vocab not a multiple of 4 or 32
    _check(ragged_vocab, 3, 32, 2, 33)


def test_max_blocks_and_large_vocab():
    ids = workload.zipf_ids(21, 255 * 64, 140000)[None]     # N = 255, the df byte's limit
    _check(ids, 255, 16, 1, 140000, idf_too=False)


@pytest.mark.parametrize("vocab", [32000, 128256])
def test_chunk4_at_128k_layouts(vocab):
    # 32768 chunk minima: with vocab 32000 they follow the df table in the
    # compact layout; with vocab 128256 they no longer fit there and the
    # general layout is used.
    ids = workload.zipf_ids(77 + vocab, 131072, vocab)[None]
    _check(ids, 16, 4, 9, vocab, idf_too=False)


def test_deterministic():
    ids = to_dev_i32(workload.make_ids(workload.CONFIGS["llama8b_32k"], batch=2))
    a = P.maxidf_summaries(ids, 8, 32, 16, 128256, return_mindf=True)
    b = P.maxidf_summaries(ids, 8, 32, 16, 128256, return_mindf=True)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("mode", [assembly.PREFIX_SUMMARY, assembly.PREFIX_ANCHOR])
def test_positions_match_eq3(mode):
    cfg = workload.CONFIGS["llama8b_32k"]
    ids = workload.make_ids(cfg, batch=2)
    sel_ref, _, _, _ = maxidf.maxidf_summaries(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab)
    sel = to_dev_i32(sel_ref)
    for i in range(cfg.num_blocks):
        pos = P.phase1_positions(sel, 2, cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk,
                                 cfg.topk, mode).cpu().numpy()
        for b in range(2):
            ref = assembly.phase1_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk,
                                            cfg.topk, sel_ref[b], mode)
            assert np.array_equal(pos[b], ref)


@pytest.mark.parametrize("L,N,sink,m,k", [
    (32768, 8, 64, 32, 16),        # sigma 512
    (3000, 3, 40, 20, 7),          # sigma 140, blocks of 1000
    (12000, 4, 5, 1, 3),           # sigma 3
    (8000, 4, 0, 1, 1),            # sigma 1: each block's first position
    (131072, 2, 64, 256, 255),     # sigma 65280: near the top of the 32-bit offset's range
    (131072, 2, 64, 256, 256),     # sigma 65536 (= Lb): the 64-bit offset
])
def test_even_spaced_positions(L, N, sink, m, k):
    # Even-Spaced prefix points j Lb + floor(p (Lb - 1) / (sigma - 1)) for
    # every block, against the oracle's map (no selection is read)
    print(f"even-spaced positions: L={L} N={N} sink={sink} m={m} k={k}", flush=True)
    for i in range(N):
        pos = P.phase1_positions(None, 1, L, N, i, sink, m, k, assembly.PREFIX_EVEN).cpu().numpy()
        ref = assembly.phase1_positions(L, N, i, sink, m, k, None, assembly.PREFIX_EVEN)
        assert np.array_equal(pos[0], ref)


def test_positions_ragged_shapes():
    L, N, s, m, k = 3 * 1000, 3, 40, 20, 7
    rng = np.random.default_rng(4)
    sel_ref = np.sort(np.stack([rng.choice(1000 // m, k, replace=False) for _ in range(N)]),
                      axis=1)[None]
    sel = to_dev_i32(sel_ref)
    for i in range(N):
        pos = P.phase1_positions(sel, 1, L, N, i, s, m, k).cpu().numpy()[0]
        assert np.array_equal(pos, assembly.phase1_positions(L, N, i, s, m, k, sel_ref[0]))
    assert math.isfinite(float(pos.sum()))


@pytest.mark.parametrize("L,N,batch,m", [(131072, 16, 600, 32), (16384, 2, 700, 16),
                                         (65536, 8, 520, 64), (131072, 4, 300, 32)])
def test_batch_beyond_compute_units(L, N, batch, m):
    # More sequences than compute units: each workgroup runs several of them
    # in turn and loads the next one's first ids while finishing the current
    # one.  Three distinct sequences repeat through the batch, so the oracle
    # runs three times and every output row is checked.
    base = np.stack([workload.zipf_ids(4000 + L // 1024 + i, L, 128256) for i in range(3)])
    print(f"maxidf persistent: batch={batch} L={L} N={N} m={m}", flush=True)
    sel_ref, mindf_ref, _, _ = maxidf.maxidf_summaries(base, N, m, 7, 128256)
    ids = base[np.arange(batch) % 3]
    sel, mindf = P.maxidf_summaries(to_dev_i32(ids), N, m, 7, 128256, return_mindf=True)
    sel, mindf = sel.cpu().numpy(), mindf.cpu().numpy()
    for r in range(3):
        assert np.array_equal(sel[r::3], np.broadcast_to(sel_ref[r], sel[r::3].shape))
        assert np.array_equal(mindf[r::3], np.broadcast_to(mindf_ref[r], mindf[r::3].shape))


@pytest.mark.parametrize("L,N,m,V,layout", [
    (32 * 1024, 32, 16, 32000, "compact bitmaps (N > 16)"),
    (64 * 2048, 64, 32, 128256, "compact bitmaps, 64 blocks"),
    (20 * 1024, 20, 32, 140000, "general bitmaps (vocab > 131072)"),
    (3 * 8192, 3, 32, 128256, "stamp code, streaming (3 rounds)"),
    (12 * 4096, 12, 16, 50000, "stamp code, streaming (blocks of 4096)"),
    (2 * 8192, 2, 8, 1000, "stamp code, resident (2 rounds)"),
])
def test_every_kernel_layout(L, N, m, V, layout):
    # one case per df-counting layout the host plan can pick
    ids = workload.zipf_ids(3000 + N + m, L, V)[None]
    print(f"maxidf layout: {layout}", flush=True)
    _check(ids, N, m, min(5, L // N // m), V)


@pytest.mark.parametrize("L,N,m,V,batch", [
    (131072, 16, 32, 128256, 16),   # the largest batch the split path takes
    (131072, 16, 32, 128256, 2),    # 32 workgroups: the largest grid whose presence is sliced
    (32768, 32, 16, 32000, 12),     # 384 workgroups: more than the chip holds at once
    (8000, 8, 4, 700, 3),           # blocks of 1000 ids: not a multiple of the workgroup
    (65536, 4, 256, 5000, 2),       # chunks of 256 ids: minima across wavefronts
    (40960, 5, 128, 145000, 1),     # a large presence table
    (4096, 2, 16, 1, 1),            # one id in the vocabulary: every df = N
    (24576, 24, 16, 32000, 3),      # 24 blocks: df bytes (more than 16 blocks), held in LDS
    (26000, 2, 8, 5000, 2),         # blocks of 13000 ids: two rounds of loads, the second partial
])
def test_split_path_shapes(L, N, m, V, batch):
    ids = np.stack([workload.zipf_ids(6000 + b + m, L, V) for b in range(min(batch, 4))])
    ids = ids[np.arange(batch) % ids.shape[0]]
    assert P.maxidf_workspace_bytes(batch, L, N, m, V) > 0
    _check(ids, N, m, min(9, L // N // m), V, idf_too=batch <= 4)


def test_split_path_large_vocab():
    # vocabularies the one-workgroup kernels do not take at this length
    ids = workload.zipf_ids(6100, 40960, 163840)[None]
    _check(ids, 5, 128, 9, 163840, single=False)
    ids = workload.zipf_ids(6101, 65536, 1000000)[None]
    _check(ids, 8, 32, 4, 1000000, single=False)
    # 24 blocks and a df byte table too large for LDS: looked up in the workspace
    ids = np.stack([workload.zipf_ids(6102 + b, 49152, 300000) for b in range(2)])
    _check(ids, 24, 32, 5, 300000, single=False)


def test_split_path_in_a_graph_replays():
    # The split path keeps no state outside the caller's workspace: captured
    # into a graph, every replay equals the eager result bit for bit, with
    # eager calls on other ids (through the same workspace) between them.
    cfg = workload.CONFIGS["llama8b_128k"]
    N, m, k, V = cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab
    ids = to_dev_i32(workload.make_ids(cfg, batch=2))
    other = to_dev_i32(np.stack([workload.zipf_ids(7000 + b, cfg.L, V) for b in range(2)]))
    ws = torch.empty(P.maxidf_workspace_bytes(2, cfg.L, N, m, V), dtype=torch.uint8, device="cuda")
    assert ws.numel() > 0
    eager = P.maxidf_summaries(ids, N, m, k, V, return_mindf=True, return_idf=True, workspace=ws)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        P.maxidf_summaries(ids, N, m, k, V, return_mindf=True, return_idf=True, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured = P.maxidf_summaries(ids, N, m, k, V, return_mindf=True, return_idf=True,
                                      workspace=ws)
    for rep in range(3):
        print(f"maxidf split graph replay {rep}", flush=True)
        for t in captured:
            t.fill_(-1)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(captured, eager):
            assert torch.equal(a.view(torch.int32), b.view(torch.int32)), f"replay {rep}"
        P.maxidf_summaries(other, N, m, k, V, return_mindf=True, workspace=ws)
        torch.cuda.synchronize()
