"""GPU parity of Phase-1 prefixed-block causal attention (and the Star anchor
baseline) against the fp64 oracle: O max-abs <= 1e-2 with relative L2 <=
1e-2, LSE max-abs <= 1e-3; retained KV bit-exact."""
import math

import numpy as np
import pytest
import torch

import paper_2607_20457_amd as P
from oracle import assembly, attention, maxidf
from paper_2607_20457_amd import workload
from tests._helpers import (check_attention, check_attention_bf16, f64, gpu_available,
                            to_dev_bf16, to_dev_i32)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _inputs(cfg, batch=1, q_scale=1.0):
    ids = workload.make_ids(cfg, batch=batch)
    q, k, v = workload.make_qkv(cfg, batch=batch, q_scale=q_scale)
    sel, _, _, _ = maxidf.maxidf_summaries(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab)
    return sel, q, k, v


def _run(cfg, i, mode, sel, q, k, v, o_dtype=P.OUT_F32, keep=False):
    print(f"phase1 parity: {cfg.name} block={i} mode={mode} q={q.shape} o_dtype={o_dtype}",
          flush=True)
    res = P.phase1_attn(to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), cfg.num_blocks, i,
                        cfg.sink, cfg.chunk, cfg.topk, None if sel is None else to_dev_i32(sel),
                        mode, o_dtype=o_dtype,
                        keep_kv=keep)
    torch.cuda.synchronize()
    return res


def _full_check(cfg, i, mode, sel, q, k, v, b=0):
    o, lse = _run(cfg, i, mode, sel, q, k, v)
    pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk,
                                    None if sel is None else sel[b], mode)
    o_ref, lse_ref = attention.phase1_attention(f64(q[b]), f64(k[b]), f64(v[b]), pos,
                                                1 / math.sqrt(cfg.d))
    check_attention(o[b].cpu().numpy(), lse[b].cpu().numpy(), o_ref, lse_ref,
                    f"{cfg.name} block {i} mode {mode}")


def _sampled_check(cfg, i, mode, sel, q, k, v, rows, b=0):
    o, lse = _run(cfg, i, mode, sel, q, k, v)
    pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk,
                                    None if sel is None else sel[b], mode)
    rows = np.array(sorted(set(int(r) for r in rows if 0 <= r < len(pos))))
    o_ref, lse_ref = attention.phase1_attention(f64(q[b]), f64(k[b]), f64(v[b]), pos,
                                                1 / math.sqrt(cfg.d), rows=rows)
    check_attention(o[b, rows].cpu().numpy(), lse[b][:, rows].cpu().numpy(), o_ref, lse_ref,
                    f"{cfg.name} block {i} mode {mode} sampled")


def test_tiny_all_blocks_full():
    cfg = workload.CONFIGS["tiny"]
    sel, q, k, v = _inputs(cfg)
    for i in range(cfg.num_blocks):
        _full_check(cfg, i, P.PREFIX_SUMMARY, sel, q, k, v)
    _full_check(cfg, 3, P.PREFIX_ANCHOR, sel, q, k, v)


@pytest.mark.parametrize("Hq,Hkv", [(8, 2), (4, 4), (16, 2)])
def test_ragged_gqa_shapes_full(Hq, Hkv):
    # n_i = 1000 + 40 + i*60: not a multiple of the 32-row or 64-key tiles
    cfg = workload.Config("ragged", L=4000, vocab=5000, num_blocks=4, sink=40, chunk=20,
                          topk=3, Hq=Hq, Hkv=Hkv, d=128, batch=2, seed=31)
    ids = workload.make_ids(cfg)
    q, k, v = workload.make_qkv(cfg)
    rng = np.random.default_rng(3)
    sel = np.sort(np.stack([[rng.choice(50, 3, replace=False) for _ in range(4)]
                            for _ in range(2)]), axis=2)
    for i in (1, 3):
        _full_check(cfg, i, P.PREFIX_SUMMARY, sel, q, k, v, b=1)
    assert ids.shape == (2, 4000)


def test_llama8b_32k_every_block_sampled():
    cfg = workload.CONFIGS["llama8b_32k"]
    sel, q, k, v = _inputs(cfg)
    for i in range(cfg.num_blocks):
        n = assembly.phase1_len(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk)
        rows = [0, 1, 63, 64, cfg.sink, cfg.sink + 1, n // 2, n - cfg.Lb - 1, n - cfg.Lb,
                n - 2, n - 1]
        _sampled_check(cfg, i, P.PREFIX_SUMMARY, sel, q, k, v, rows)


def test_llama8b_128k_block15_sampled():
    # the full-size headline launch: block 15 of 16, n = 23616
    cfg = workload.CONFIGS["llama8b_128k"]
    sel, q, k, v = _inputs(cfg)
    n = assembly.phase1_len(cfg.L, 16, 15, cfg.sink, cfg.chunk, cfg.topk)
    assert n == 23616
    rng = np.random.default_rng(15)
    rows = [0, 63, 64, 65, 1087, 1088, 15423, 15424, n - 1] + list(rng.integers(0, n, 8))
    _sampled_check(cfg, 15, P.PREFIX_SUMMARY, sel, q, k, v, rows)
    _sampled_check(cfg, 15, P.PREFIX_ANCHOR, sel, q, k, v, [0, 8191, 8192, 16383])


def test_peaked_attention_control():
    # Q scaled by 8: softmax mass concentrates, |O| ~ 1, so a zero or shifted
    # output cannot pass the absolute tolerance
    cfg = workload.Config("peaked", L=8192, vocab=4000, num_blocks=4, sink=64, chunk=32,
                          topk=8, Hq=8, Hkv=2, d=128, seed=41)
    sel, q, k, v = _inputs(cfg, q_scale=8.0)
    o, _ = _run(cfg, 2, P.PREFIX_SUMMARY, sel, q, k, v)
    assert float(o.abs().mean()) > 0.2
    _full_check(cfg, 2, P.PREFIX_SUMMARY, sel, q, k, v)


def test_bf16_output_and_kept_kv():
    cfg = workload.CONFIGS["tiny"]
    sel, q, k, v = _inputs(cfg)
    o32, lse32 = _run(cfg, 2, P.PREFIX_SUMMARY, sel, q, k, v)
    o16, lse16, kk, vk = _run(cfg, 2, P.PREFIX_SUMMARY, sel, q, k, v, o_dtype=P.OUT_BF16,
                              keep=True)
    # bf16 output is the fp32 output rounded once (half an ulp of bf16)
    ref = o32.to(torch.bfloat16)
    assert torch.equal(o16, ref)
    assert torch.equal(lse16, lse32)
    Lb = cfg.Lb
    assert torch.equal(kk.cpu().view(torch.int16),
                       torch.from_numpy(k[:, 2 * Lb:3 * Lb].view(np.int16)))
    assert torch.equal(vk.cpu().view(torch.int16),
                       torch.from_numpy(v[:, 2 * Lb:3 * Lb].view(np.int16)))


def test_degenerate_sink_and_k_zero():
    cfg = workload.Config("deg", L=2048, vocab=1000, num_blocks=4, sink=0, chunk=16, topk=0,
                          Hq=4, Hkv=1, d=64, seed=51)
    q, k, v = workload.make_qkv(cfg)
    sel = np.zeros((1, 4, 0), dtype=np.int32)
    _full_check(cfg, 3, P.PREFIX_SUMMARY, sel, q, k, v)


def test_deterministic():
    cfg = workload.CONFIGS["tiny"]
    sel, q, k, v = _inputs(cfg)
    a = _run(cfg, 3, P.PREFIX_SUMMARY, sel, q, k, v)
    b = _run(cfg, 3, P.PREFIX_SUMMARY, sel, q, k, v)
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def _bits_equal(a, b):
    return a.shape == b.shape and torch.equal(a.contiguous().view(torch.int32),
                                              b.contiguous().view(torch.int32))


def test_causal_launches_on_several_streams():
    # Causal launches take a work-counter slot per stream and may run at the
    # same time on different streams: each must equal its result alone,
    # bit for bit, on every repetition (the counters start from zero again).
    cfg = workload.CONFIGS["llama8b_32k"]
    sel, q, k, v = _inputs(cfg)
    Q, K, V, S = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), to_dev_i32(sel)
    blocks = [7, 6, 5, 4]
    run = lambda i: P.phase1_attn(Q, K, V, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S)
    ref = [run(i) for i in blocks]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream() for _ in blocks]
    for rep in range(3):
        print(f"several streams: repetition {rep}", flush=True)
        outs = []
        for i, s in zip(blocks, streams):
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                outs.append(run(i))
        torch.cuda.synchronize()
        for (o, lse), (o_r, lse_r), i in zip(outs, ref, blocks):
            assert _bits_equal(o, o_r) and _bits_equal(lse, lse_r), f"block {i}"


def test_causal_launches_beyond_the_counter_slots():
    # 70 streams of their own (more than the 64 counter slots of a device):
    # the first streams get a slot, the rest the plain launch; every result
    # equals the one on the default stream, bit for bit.
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime this process already uses
    hip.hipStreamCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
    cfg = workload.CONFIGS["tiny"]
    sel, q, k, v = _inputs(cfg)
    Q, K, V, S = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), to_dev_i32(sel)
    i = 3
    o_ref, lse_ref = P.phase1_attn(Q, K, V, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S)
    torch.cuda.synchronize()
    handles = []
    try:
        for n in range(70):
            h = ctypes.c_void_p()
            assert hip.hipStreamCreate(ctypes.byref(h)) == 0
            handles.append(h)
            with torch.cuda.stream(torch.cuda.ExternalStream(h.value)):
                o, lse = P.phase1_attn(Q, K, V, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S)
            torch.cuda.synchronize()
            assert _bits_equal(o, o_ref) and _bits_equal(lse, lse_ref), f"stream {n}"
    finally:
        torch.cuda.synchronize()
        for h in handles:
            hip.hipStreamDestroy(h)


def test_causal_launch_in_a_graph_replays():
    # Captured into a graph the causal launch takes the one-workgroup-per-item
    # form; every replay, with eager launches between them, must equal the
    # eager result bit for bit.
    cfg = workload.CONFIGS["llama8b_32k"]
    sel, q, k, v = _inputs(cfg)
    Q, K, V, S = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), to_dev_i32(sel)
    i = 5
    n = P.phase1_len(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk)
    o_eager, lse_eager = P.phase1_attn(Q, K, V, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S)
    O = torch.empty((1, n, cfg.Hq, cfg.d), dtype=torch.float32, device="cuda")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up outside the capture
        P.phase1_attn(Q, K, V, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S, out=O)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _, lse_g = P.phase1_attn(Q, K, V, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S,
                                 out=O)
    for rep in range(3):
        print(f"graph replay {rep}", flush=True)
        O.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert _bits_equal(O, o_eager) and _bits_equal(lse_g, lse_eager), f"replay {rep}"
        # eager work between the replays, on the same stream
        o2, _ = P.phase1_attn(Q, K, V, cfg.num_blocks, i - 1, cfg.sink, cfg.chunk, cfg.topk, S)
        torch.cuda.synchronize()


def test_far_larger_later_score_takes_exact_pass():
    # A key placed after the first 32 keys whose score exceeds the first keys'
    # maximum by far more than 2^64 in weight: the reference-max pass flags
    # it and the exact online-softmax pass must give the oracle's answer.
    cfg = workload.Config("spike", L=2048, vocab=1000, num_blocks=2, sink=16, chunk=16,
                          topk=2, Hq=4, Hkv=1, d=64, seed=61)
    q, k, v = workload.make_qkv(cfg)
    qf = workload.bf16_bits_to_f32(q) + 1.0          # queries share a mean direction
    q = workload.f32_to_bf16_bits(qf)
    kf = workload.bf16_bits_to_f32(k)
    kf[0, 500] = 10.0                                # q.k / sqrt(d) ~ 80 for that key
    k = workload.f32_to_bf16_bits(kf)
    sel = np.array([[[0, 5], [1, 2]]], dtype=np.int32)
    _full_check(cfg, 0, P.PREFIX_SUMMARY, sel, q, k, v)
    _full_check(cfg, 1, P.PREFIX_SUMMARY, sel, q, k, v)


def test_even_spaced_prefix_tiny_full():
    # Even-Spaced baseline: Sigma_j = k*m evenly spaced tokens of B_j
    cfg = workload.CONFIGS["tiny"]
    sel, q, k, v = _inputs(cfg)
    for i in range(cfg.num_blocks):
        _full_check(cfg, i, P.PREFIX_EVEN, None, q, k, v)


def test_even_spaced_prefix_128k_block15_sampled():
    cfg = workload.CONFIGS["llama8b_128k"]
    _, q, k, v = _inputs(cfg)
    n = P.phase1_len(cfg.L, cfg.num_blocks, 15, cfg.sink, cfg.chunk, cfg.topk, P.PREFIX_EVEN)
    sigma = cfg.topk * cfg.chunk
    rows = [0, 63, 64, 64 + sigma - 1, 64 + sigma, 64 + 7 * sigma + 5, n - 8193, n - 8192,
            n - 1] + list(np.random.default_rng(3).integers(0, n, 120))
    _sampled_check(cfg, 15, P.PREFIX_EVEN, None, q, k, v, rows)


@pytest.mark.parametrize("Lb,sink,m,k", [(1024, 64, 16, 4), (1000, 10, 20, 7), (4096, 0, 32, 16),
                                         (777, 5, 1, 1), (256, 3, 8, 0)])
def test_even_spaced_positions_match_the_oracle(Lb, sink, m, k):
    N = 5
    for i in range(N):
        pos = P.phase1_positions(None, 2, N * Lb, N, i, sink, m, k, P.PREFIX_EVEN,
                                 device="cuda").cpu().numpy()
        ref = assembly.phase1_positions(N * Lb, N, i, sink, m, k, None, assembly.PREFIX_EVEN)
        assert np.array_equal(pos[0], ref) and np.array_equal(pos[1], ref)


def _oracle_rows(cfg, i, mode, sel_b, q_b, k_b, v_b, rows, topk=None):
    topk = cfg.topk if topk is None else topk
    pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk, topk,
                                    sel_b, mode)
    rows = np.array(sorted(set(int(r) for r in rows if 0 <= r < len(pos))))
    # fp64 copies of only the positions the sampled rows read (np.zeros
    # commits no memory for the rest)
    qp, kp = pos[rows], pos[:rows.max() + 1]
    Qf, Kf, Vf = np.zeros(q_b.shape), np.zeros(k_b.shape), np.zeros(v_b.shape)
    Qf[qp], Kf[kp], Vf[kp] = f64(q_b[qp]), f64(k_b[kp]), f64(v_b[kp])
    o_ref, _ = attention.phase1_attention(Qf, Kf, Vf, pos, 1 / math.sqrt(cfg.d), rows=rows)
    return rows, o_ref


def test_llama8b_128k_block15_bench_launch_no_lse():
    # Exactly the launch the benchmark times: block 15 of 16, fp32 O into a
    # caller buffer, no LSE (the kernel build without the fp32 weight sum),
    # with the retained KV(B_15) copied out; then the Even-Spaced and Star
    # launches the benchmark times the same way.
    cfg = workload.CONFIGS["llama8b_128k"]
    sel, q, k, v = _inputs(cfg)
    N, i = cfg.num_blocks, cfg.num_blocks - 1
    n = P.phase1_len(cfg.L, N, i, cfg.sink, cfg.chunk, cfg.topk)
    Q, K, V, S = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), to_dev_i32(sel)
    O = torch.empty((1, n, cfg.Hq, cfg.d), dtype=torch.float32, device="cuda")
    print(f"phase1 bench launch: {cfg.name} block {i} n={n} no LSE, keep KV", flush=True)
    res = P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, cfg.topk, S, out=O,
                        return_lse=False, keep_kv=True)
    torch.cuda.synchronize()
    assert res[0] is O and len(res) == 3
    Kk, Vk = res[1], res[2]
    rng = np.random.default_rng(151)
    rows = [0, 63, 64, 65, 1087, 1088, 15423, 15424, n - 8193, n - 8192, n - 2, n - 1] + \
        list(rng.integers(0, n, 40))
    rows, o_ref = _oracle_rows(cfg, i, P.PREFIX_SUMMARY, sel[0], q[0], k[0], v[0], rows)
    check_attention(O[0, rows].cpu().numpy(), None, o_ref, None, "128K block 15, no LSE")
    # KV(B_15): the last Lb rows of Input_15 are block 15's own tokens, bit for bit
    Lb = cfg.Lb
    assert torch.equal(Kk.cpu().view(torch.int16),
                       torch.from_numpy(k[:, i * Lb:(i + 1) * Lb].view(np.int16)))
    assert torch.equal(Vk.cpu().view(torch.int16),
                       torch.from_numpy(v[:, i * Lb:(i + 1) * Lb].view(np.int16)))
    # no-LSE and LSE builds give the same O
    o_lse, _ = P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, cfg.topk, S)
    torch.cuda.synchronize()
    d = (o_lse[0, rows] - O[0, rows]).abs().max().item()
    assert d <= 1e-3, d
    del o_lse
    for mode in (P.PREFIX_EVEN, P.PREFIX_ANCHOR):
        n_m = P.phase1_len(cfg.L, N, i, cfg.sink, cfg.chunk, cfg.topk, mode)
        Om = torch.empty((1, n_m, cfg.Hq, cfg.d), dtype=torch.float32, device="cuda")
        print(f"phase1 bench launch: mode {mode} n={n_m} no LSE", flush=True)
        P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, cfg.topk, None, mode, out=Om,
                      return_lse=False)
        torch.cuda.synchronize()
        rows_m = [0, 63, 64, 8191, 8192, n_m - 8193, n_m - 1] + list(rng.integers(0, n_m, 20))
        rows_m, o_ref = _oracle_rows(cfg, i, mode, None, q[0], k[0], v[0], rows_m)
        check_attention(Om[0, rows_m].cpu().numpy(), None, o_ref, None,
                        f"128K block 15 mode {mode}, no LSE")


_SWEEP = {}


def _sweep_inputs():
    # batch 4 x 131072 tokens of the 8B layer (the anchor-vs-Pulsar sweep)
    if not _SWEEP:
        cfg = workload.CONFIGS["sweep_128k_b4"]
        ids = workload.make_ids(cfg)
        q, k, v = workload.make_qkv(cfg)
        _SWEEP.update(cfg=cfg, ids=ids, q=q, k=k, v=v, Q=to_dev_bf16(q), K=to_dev_bf16(k),
                      V=to_dev_bf16(v))
    return _SWEEP


@pytest.mark.parametrize("topk", [8, 64])
def test_sweep_batch4_bf16_no_lse(topk):
    # The sweep's launches: batch 4, bf16 O, no LSE, top-k 8 and 64 (at 64,
    # block 15 has n = 38976 rows and a 960-run table); rows sampled from two
    # sequences of the batch, selection checked bit for bit first.
    w = _sweep_inputs()
    cfg = w["cfg"]
    N = cfg.num_blocks
    sel = P.maxidf_summaries(torch.from_numpy(w["ids"]).cuda(), N, cfg.chunk, topk, cfg.vocab)
    torch.cuda.synchronize()
    sel_ref, _, _, _ = maxidf.maxidf_summaries(w["ids"], N, cfg.chunk, topk, cfg.vocab)
    assert np.array_equal(sel.cpu().numpy(), sel_ref)
    rng = np.random.default_rng(topk)
    for i in (1, 8, N - 1):
        n = P.phase1_len(cfg.L, N, i, cfg.sink, cfg.chunk, topk)
        O = torch.empty((cfg.batch, n, cfg.Hq, cfg.d), dtype=torch.bfloat16, device="cuda")
        print(f"sweep launch: batch {cfg.batch} block {i} top-k {topk} n={n} bf16 no LSE",
              flush=True)
        P.phase1_attn(w["Q"], w["K"], w["V"], N, i, cfg.sink, cfg.chunk, topk, sel,
                      o_dtype=P.OUT_BF16, return_lse=False, out=O)
        torch.cuda.synchronize()
        for b in (1, 3):
            rows = [0, 63, 64, n - cfg.Lb - 1, n - cfg.Lb, n - 1] + list(rng.integers(0, n, 10))
            rows, o_ref = _oracle_rows(cfg, i, P.PREFIX_SUMMARY, sel_ref[b], w["q"][b], w["k"][b],
                                       w["v"][b], rows, topk=topk)
            check_attention_bf16(O[b, rows].float().cpu().numpy(), o_ref,
                                 f"sweep b={b} block {i} k={topk}")
        del O


def test_sweep_batch4_anchor_bf16_no_lse():
    w = _sweep_inputs()
    cfg = w["cfg"]
    N = cfg.num_blocks
    rng = np.random.default_rng(5)
    for i in (1, N - 1):
        n = P.phase1_len(cfg.L, N, i, cfg.sink, cfg.chunk, 0, P.PREFIX_ANCHOR)
        O = torch.empty((cfg.batch, n, cfg.Hq, cfg.d), dtype=torch.bfloat16, device="cuda")
        print(f"sweep anchor launch: batch {cfg.batch} block {i} n={n} bf16 no LSE", flush=True)
        P.phase1_attn(w["Q"], w["K"], w["V"], N, i, cfg.sink, cfg.chunk, 0, None,
                      P.PREFIX_ANCHOR, o_dtype=P.OUT_BF16, return_lse=False, out=O)
        torch.cuda.synchronize()
        for b in (0, 2):
            rows = [0, 8191, 8192, n - 1] + list(rng.integers(0, n, 8))
            rows, o_ref = _oracle_rows(cfg, i, P.PREFIX_ANCHOR, None, w["q"][b], w["k"][b],
                                       w["v"][b], rows, topk=0)
            check_attention_bf16(O[b, rows].float().cpu().numpy(), o_ref,
                                 f"sweep anchor b={b} block {i}")
        del O
    _SWEEP.clear()
