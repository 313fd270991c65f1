"""Benchmark of the Pulsar Attention hot path on one MI355X.

One step = one pass of the whole path over one 131072-token sequence of the
Llama-3.1-8B-shaped layer (32 query / 8 KV heads, head_dim 128, bf16):

  1. Max-IDF summaries over all 16 blocks of 8192 tokens (df, chunk min-df,
     top-32 chunks of 32 tokens per block);
  2. Phase-1 prefixed-block causal attention for block 15, the longest input
     (n = 8192 + 64 + 15 * 1024 = 23616 rows), with the Eq. 3 gather fused
     into the kernel's loads, and the retained KV(B_15) copied out;
  3. Phase-2 partial attention of 64 query tokens over the 16 retained
     shards of 8192 keys, and the online-softmax merge.

Inputs are synthetic (Zipf(1.1) ids over 128256, bf16 N(0,1) Q/K/V) and
already resident in HBM when timing starts.  The JSON line reports the Phase-1
attention FLOP rate of block 15 as ``value`` (the metric), per-kernel rates
measured with HIP events on the launch stream, the roofline of that dominant
kernel (bf16 MFMA bound), the Star Attention anchor baseline for the same
block, the anchor-vs-Pulsar sweep (batch 4 x 128K, all 16 blocks, top-k
8/32/64) beside the cost model's ratios, Max-IDF at batch 8 and 1024, and the
fp64 CPU oracle timed on a bounded sample.

``--profile-step`` runs only the warm-up and timed steps (for profiler
traces whose rows then hold the step's launches alone).  ``--sweep`` prints
the anchor-vs-Pulsar sweep and a wider Max-IDF batch sweep instead.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import subprocess
import sys
import threading
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2607_20457_amd as P  # noqa: E402
from paper_2607_20457_amd import workload  # noqa: E402

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak (published)
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E peak (published)
# the attention kernel's sources: the HBM-traffic figure is used only while
# they are unchanged since the counters were taken
ATTN_SRCS = [os.path.join(ROOT, "paper_2607_20457_amd", "csrc", f)
             for f in ("attn_kernel.hpp", "attn.hip", "attn_d128.hip", "common.hpp")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def causal_flops(n, Hq, d):
    return 4 * d * Hq * n * (n + 1) // 2


def full_flops(nq, nk, Hq, d):
    return 4 * d * Hq * nq * nk


def bf16_dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def src_sha(paths):
    h = hashlib.sha256()
    for path in paths:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel_key):
    """HBM bytes per launch from the committed rocprofv3 PMC summary, or None
    if the kernel source changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)[kernel_key]
    except (OSError, KeyError, ValueError):
        return None
    if t.get("source_sha") != src_sha(ATTN_SRCS):
        return None
    return t.get("bytes_per_launch")


# GPU clock cycles of the spin kernel that precedes a short timed call
SPIN_CYCLES = 400_000


class Timer:
    """HIP events on the current stream around each launch of one kernel.
    spin=True first queues a short spin kernel, so that the host has queued
    the timed call before its start event runs: the events then bracket the
    device's time alone, not the host's launch overhead (which otherwise
    dominates calls of a few microseconds)."""

    def __init__(self, spin: bool = False):
        self.pairs = []
        self.spin = spin

    def __enter__(self):
        self.s = torch.cuda.Event(enable_timing=True)
        self.e = torch.cuda.Event(enable_timing=True)
        if self.spin:
            torch.cuda._sleep(SPIN_CYCLES)
        self.s.record()
        return self

    def __exit__(self, *exc):
        self.e.record()
        self.pairs.append((self.s, self.e))

    def mean_ms(self):
        return sum(s.elapsed_time(e) for s, e in self.pairs) / max(1, len(self.pairs))


def cpu_oracle_baseline(ids, q, k, v, sel_ref, cfg, n, budget_s=15.0):
    """The fp64 oracle on a bounded sample: Max-IDF over the whole sequence,
    then Phase-1 attention for evenly spread rows of block 15 until the
    budget is used.  Returns a cpu_baseline dict in TFLOP/s."""
    from oracle import assembly, attention, maxidf
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: report the affinity size
        blas_threads = len(os.sched_getaffinity(0))
    t0 = time.perf_counter()
    maxidf.maxidf_summaries(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab)
    t_idf = time.perf_counter() - t0
    pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, cfg.num_blocks - 1, cfg.sink,
                                    cfg.chunk, cfg.topk, sel_ref[0])
    f64 = lambda x: workload.bf16_bits_to_f32(x).astype(np.float64)
    Q, K, V = f64(q[0]), f64(k[0]), f64(v[0])
    scale = 1 / math.sqrt(cfg.d)
    rows_all = np.linspace(0, n - 1, 2048).astype(np.int64)[::-1]  # longest rows first
    flops, done, t_attn = 0, 0, 0.0
    for b0 in range(0, rows_all.size, 8):
        rows = rows_all[b0:b0 + 8]
        t0 = time.perf_counter()
        attention.phase1_attention(Q, K, V, pos, scale, rows=rows)
        t_attn += time.perf_counter() - t0
        flops += sum(4 * cfg.d * cfg.Hq * (int(r) + 1) for r in rows)
        done += rows.size
        if t_attn > budget_s:
            break
    return {
        "value": flops / t_attn / 1e12,
        "unit": "TFLOP/s",
        "cores": int(blas_threads),
        "kind": "oracle",
        "sample": f"fp64 Phase-1 attention for {done} of the 23616 rows of block 15 (all 32 "
                  f"heads, rows evenly spread, {t_attn:.1f} s); Max-IDF oracle over the full "
                  f"131072-token sequence took {t_idf:.2f} s "
                  f"({cfg.L / t_idf:.3g} tokens/s, 1 core, pure Python)",
        "maxidf_tokens_per_s": cfg.L / t_idf,
    }


def calibration_copy():
    """A plain device copy of a known size (1 GiB read, 1 GiB write), far
    larger than the caches: the scale for the FETCH_SIZE / WRITE_SIZE counters
    of a rocprofv3 --pmc run of this command.  Returns the bytes copied."""
    src = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    return src.numel() * 4


IDF_THROUGHPUT_BATCH = 1024
METRIC = "Phase-1 prefixed-block attn TFLOP/s (% bf16 MFMA peak); Max-IDF tokens/s"


def run_main(args):
    cfg = workload.CONFIGS["llama8b_128k"]
    N, i_last = cfg.num_blocks, cfg.num_blocks - 1
    ids = workload.make_ids(cfg, batch=1)
    q, k, v = workload.make_qkv(cfg, batch=1)
    Tq = 64
    q2 = workload.bf16_normal(cfg.seed * 10 + 7, (Tq, cfg.Hq, cfg.d))
    d_ids = torch.from_numpy(ids).cuda()
    Q, K, V = bf16_dev(q), bf16_dev(k), bf16_dev(v)
    q_dev = bf16_dev(q2)
    n = P.phase1_len(cfg.L, N, i_last, cfg.sink, cfg.chunk, cfg.topk)
    n_star = P.phase1_len(cfg.L, N, i_last, cfg.sink, cfg.chunk, cfg.topk, P.PREFIX_ANCHOR)
    O = torch.empty((1, n, cfg.Hq, cfg.d), dtype=torch.float32, device="cuda")
    O_star = torch.empty((1, n_star, cfg.Hq, cfg.d), dtype=torch.float32, device="cuda")
    ws = torch.empty(P.phase2_workspace_bytes(N, Tq, cfg.Lb, cfg.Hq, cfg.Hkv, cfg.d) or 1,
                     dtype=torch.uint8, device="cuda")
    idf_ws = torch.empty(max(P.maxidf_workspace_bytes(1, cfg.L, N, cfg.chunk, cfg.vocab), 16),
                         dtype=torch.uint8, device="cuda")
    t_idf, t_p1, t_p2, t_star = Timer(), Timer(), Timer(), Timer(spin=True)

    def step(timed):
        with (t_idf if timed else _Null()):
            sel = P.maxidf_summaries(d_ids, N, cfg.chunk, cfg.topk, cfg.vocab, workspace=idf_ws)
        with (t_p1 if timed else _Null()):
            # the forward pass yields O for every row and the retained KV(B_15);
            # no LSE is needed downstream of Phase 1
            P.phase1_attn(Q, K, V, N, i_last, cfg.sink, cfg.chunk, cfg.topk, sel, out=O,
                          return_lse=False, keep_kv=True)
        with (t_p2 if timed else _Null()):
            shards_k = K[0].view(N, cfg.Lb, cfg.Hkv, cfg.d)
            shards_v = V[0].view(N, cfg.Lb, cfg.Hkv, cfg.d)
            o_parts, lse_parts = P.phase2_partial(q_dev, shards_k, shards_v, workspace=ws)
            P.lse_merge(o_parts, lse_parts)
        return sel

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        sel = step(True)
    end.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(end) / args.steps

    f_p1 = causal_flops(n, cfg.Hq, cfg.d)
    f_p2 = full_flops(Tq, N * cfg.Lb, cfg.Hq, cfg.d)
    p1_ms = t_p1.mean_ms()
    p1_tflops = f_p1 / (p1_ms * 1e-3) / 1e12
    if args.profile_step:
        if args.calibrate:
            calibration_copy()
        print(json.dumps({"metric": METRIC, "value": p1_tflops, "unit": "TFLOP/s",
                          "ms_per_step": ms_step, "phase1_attn_ms": p1_ms,
                          "phase2_partial_merge_ms": t_p2.mean_ms(),
                          "maxidf_ms": t_idf.mean_ms(), "steps": args.steps,
                          "warmup": args.warmup}), flush=True)
        return

    # Star Attention anchor baseline for the same block, timed the same way
    for _ in range(2):
        P.phase1_attn(Q, K, V, N, i_last, cfg.sink, cfg.chunk, cfg.topk, None, P.PREFIX_ANCHOR,
                      out=O_star, return_lse=False)
    for _ in range(args.steps):
        with t_star:
            P.phase1_attn(Q, K, V, N, i_last, cfg.sink, cfg.chunk, cfg.topk, None,
                          P.PREFIX_ANCHOR, out=O_star, return_lse=False)
    torch.cuda.synchronize()

    # Max-IDF throughput: 1024 sequences of 128K ids (512 MiB of ids), every
    # compute unit busy; the batch-1 call in the step is latency-bound on one
    t_idf_big = Timer(spin=True)
    big = d_ids.expand(IDF_THROUGHPUT_BATCH, cfg.L).contiguous()
    P.maxidf_summaries(big, N, cfg.chunk, cfg.topk, cfg.vocab)
    for _ in range(5):
        with t_idf_big:
            P.maxidf_summaries(big, N, cfg.chunk, cfg.topk, cfg.vocab)
    torch.cuda.synchronize()
    del big

    # The other chunk scorers over the same sequence (batch 1, latency-bound
    # on one compute unit) and over 256 copies of it (one per compute unit)
    scorer_rows = {}
    big = d_ids.expand(256, cfg.L).contiguous()
    for name, sc in (("tfidf", P.SCORE_TFIDF), ("bm25", P.SCORE_BM25),
                     ("entropy", P.SCORE_ENTROPY)):
        row = {}
        for batch, inp in ((1, d_ids), (256, big)):
            t = Timer(spin=True)
            P.chunk_summaries(inp, N, cfg.chunk, cfg.topk, cfg.vocab, sc)
            for _ in range(5):
                with t:
                    P.chunk_summaries(inp, N, cfg.chunk, cfg.topk, cfg.vocab, sc)
            torch.cuda.synchronize()
            row[f"batch{batch}_ms"] = t.mean_ms()
            row[f"batch{batch}_tokens_per_s"] = batch * cfg.L / (t.mean_ms() * 1e-3)
        scorer_rows[name] = row
    del big

    # Phase 1 of block 15 with the Even-Spaced baseline prefix (same row count)
    t_even = Timer(spin=True)
    for _ in range(2):
        P.phase1_attn(Q, K, V, N, i_last, cfg.sink, cfg.chunk, cfg.topk, None, P.PREFIX_EVEN,
                      out=O, return_lse=False)
    for _ in range(5):
        with t_even:
            P.phase1_attn(Q, K, V, N, i_last, cfg.sink, cfg.chunk, cfg.topk, None,
                          P.PREFIX_EVEN, out=O, return_lse=False)
    torch.cuda.synchronize()

    # Rotary embedding of the layer's Q and K at their global positions (the
    # sparse-position mode), once per layer for the whole context; on copies,
    # so that the attention inputs above stay as drawn
    t_rope = Timer(spin=True)
    Qr, Kr = Q.clone(), K.clone()
    P.rope_(Qr)
    P.rope_(Kr)
    for _ in range(5):
        with t_rope:
            P.rope_(Qr)
            P.rope_(Kr)
    torch.cuda.synchronize()
    rope_bytes = 2 * (Qr.numel() + Kr.numel()) * 2
    del Qr, Kr

    # Phase 2 of new tokens over the 16 retained shards: the 64-token query
    # encoding (its own rows causally), and one decode step (1 token after 64)
    kg = bf16_dev(workload.bf16_normal(cfg.seed * 10 + 8, (Tq + 1, cfg.Hkv, cfg.d)))
    vg = bf16_dev(workload.bf16_normal(cfg.seed * 10 + 9, (Tq + 1, cfg.Hkv, cfg.d)))
    shards_k = K[0].view(N, cfg.Lb, cfg.Hkv, cfg.d)
    shards_v = V[0].view(N, cfg.Lb, cfg.Hkv, cfg.d)
    q_dec = q_dev[:1].contiguous()
    t_enc, t_dec = Timer(spin=True), Timer(spin=True)
    for _ in range(2):
        P.phase2_query(q_dev, kg[:Tq], vg[:Tq], 0, shards_k, shards_v)
        P.phase2_query(q_dec, kg, vg, Tq, shards_k, shards_v)
    for _ in range(5):
        with t_enc:
            P.phase2_query(q_dev, kg[:Tq], vg[:Tq], 0, shards_k, shards_v)
        with t_dec:
            P.phase2_query(q_dec, kg, vg, Tq, shards_k, shards_v)
    torch.cuda.synchronize()
    kv_bytes = 2 * N * cfg.Lb * cfg.Hkv * cfg.d * 2

    # Max-IDF at batch 8 (the sweep's setting): latency-bound, 8 compute units
    t_idf8 = Timer(spin=True)
    ids8 = workload.make_ids(workload.CONFIGS["sweep_128k_b4"], batch=8)
    d_ids8 = torch.from_numpy(ids8).cuda()
    ws8 = torch.empty(max(P.maxidf_workspace_bytes(8, cfg.L, N, cfg.chunk, cfg.vocab), 16),
                      dtype=torch.uint8, device="cuda")
    P.maxidf_summaries(d_ids8, N, cfg.chunk, cfg.topk, cfg.vocab, workspace=ws8)
    for _ in range(5):
        with t_idf8:
            P.maxidf_summaries(d_ids8, N, cfg.chunk, cfg.topk, cfg.vocab, workspace=ws8)
    torch.cuda.synchronize()

    f_star = causal_flops(n_star, cfg.Hq, cfg.d)
    p2_ms, idf_ms, star_ms = t_p2.mean_ms(), t_idf.mean_ms(), t_star.mean_ms()
    idf_bytes = cfg.L * 4 + N * cfg.topk * 4
    p2_bytes = 2 * N * cfg.Lb * cfg.Hkv * cfg.d * 2 + Tq * cfg.Hq * cfg.d * 2 \
        + 2 * N * Tq * cfg.Hq * (cfg.d + 1) * 4
    sweep = None
    if not args.no_sweep:
        del O, O_star
        torch.cuda.empty_cache()
        sweep, _ = cfg5_sweep(reps=2)
    result = {
        "metric": METRIC,
        "value": p1_tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: Zipf(1.1) token ids over vocab 128256, bf16 N(0,1) Q/K/V, "
                "random-init single layer",
        "config": {"workload": "Llama-3.1-8B-shaped layer, 128K context (131072 tokens, batch 1), "
                               "16 blocks x 8192, sink 64, chunk 32, top-k 32; Phase-1 for block 15 "
                               "(23616 rows); Phase-2 for 64 query tokens over 16 shards x 8192",
                   "Hq": cfg.Hq, "Hkv": cfg.Hkv, "head_dim": cfg.d, "seq_len": cfg.L,
                   "batch": 1, "parallelism": "single GPU"},
        "kernels": {
            "step_attn_tflops": (f_p1 + f_p2) / (ms_step * 1e-3) / 1e12,
            "phase1_attn_ms": p1_ms,
            "phase1_attn_tflops": p1_tflops,
            "phase1_pct_bf16_peak": 100 * p1_tflops / PEAK_BF16_TFLOPS,
            "maxidf_ms": idf_ms,
            "maxidf_tokens_per_s": cfg.L / (idf_ms * 1e-3),
            "maxidf_gbps_algorithmic": idf_bytes / (idf_ms * 1e-3) / 1e9,
            "maxidf_batch8": {
                "ms": t_idf8.mean_ms(),
                "tokens_per_s": 8 * cfg.L / (t_idf8.mean_ms() * 1e-3),
                "gbps_algorithmic": 8 * idf_bytes / (t_idf8.mean_ms() * 1e-3) / 1e9,
            },
            "maxidf_throughput": {
                "batch": IDF_THROUGHPUT_BATCH,
                "ms": t_idf_big.mean_ms(),
                "tokens_per_s": IDF_THROUGHPUT_BATCH * cfg.L / (t_idf_big.mean_ms() * 1e-3),
                "gbps_algorithmic": IDF_THROUGHPUT_BATCH * idf_bytes / (t_idf_big.mean_ms() * 1e-3) / 1e9,
                "pct_hbm_peak": 100 * IDF_THROUGHPUT_BATCH * idf_bytes / (t_idf_big.mean_ms() * 1e-3)
                                / 1e9 / PEAK_HBM_GBPS,
            },
            "rope_qk": {
                "ms": t_rope.mean_ms(),
                "gbps_algorithmic": rope_bytes / (t_rope.mean_ms() * 1e-3) / 1e9,
                "pct_hbm_peak": 100 * rope_bytes / (t_rope.mean_ms() * 1e-3) / 1e9 / PEAK_HBM_GBPS,
            },
            "phase2_query": {
                "encoding_tq64_ms": t_enc.mean_ms(),
                "decode_step_ms": t_dec.mean_ms(),
                "decode_kv_gbps": kv_bytes / (t_dec.mean_ms() * 1e-3) / 1e9,
                "decode_pct_hbm_peak": 100 * kv_bytes / (t_dec.mean_ms() * 1e-3) / 1e9 / PEAK_HBM_GBPS,
            },
            "scorers": scorer_rows,
            "even_spaced_phase1_ms": t_even.mean_ms(),
            "phase2_partial_merge_ms": p2_ms,
            "phase2_tflops": f_p2 / (p2_ms * 1e-3) / 1e12,
            "phase2_gbps_algorithmic": p2_bytes / (p2_ms * 1e-3) / 1e9,
        },
        "star_anchor": {
            "n_rows": n_star, "ms": star_ms,
            "tflops": f_star / (star_ms * 1e-3) / 1e12,
            "flop_ratio_star_over_pulsar": f_star / f_p1,
            "time_ratio_star_over_pulsar": star_ms / p1_ms,
        },
        "sweep_cfg5": sweep,
        "roofline": {
            "bound": "mfma",
            "achieved": p1_tflops,
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": p1_tflops / PEAK_BF16_TFLOPS,
            "traffic": measured_traffic("attn_phase1_128k_block15"),
        },
    }
    if args.calibrate:
        result["calibration_copy_bytes"] = calibration_copy()
    if not args.no_cpu:
        from oracle import maxidf as oracle_maxidf
        sel_ref, _, _, _ = oracle_maxidf.maxidf_summaries(ids, N, cfg.chunk, cfg.topk, cfg.vocab)
        assert np.array_equal(sel.cpu().numpy(), sel_ref), "selection differs from the oracle"
        result["cpu_baseline"] = cpu_oracle_baseline(ids, q, k, v, sel_ref, cfg, n,
                                                     budget_s=args.cpu_budget)
    print(json.dumps(result), flush=True)


# Star/Pulsar Phase-1 FLOP ratios of the cost model (F(n) proportional to n^2,
# Table 4's accounting) at 16 blocks of 8192, sink 64, chunk 32: the last
# block and the sum over all 16 blocks, per top-k
def model_ratios(topk, L=131072, N=16, sink=64, chunk=32):
    Lb = L // N
    star = [Lb] + [2 * Lb] * (N - 1)
    pul = [Lb] + [Lb + sink + i * topk * chunk for i in range(1, N)]
    return (star[-1] ** 2 / pul[-1] ** 2,
            sum(x * x for x in star) / sum(x * x for x in pul))


def cfg5_sweep(reps=3):
    """Anchor vs Pulsar Phase-1 over all 16 blocks, batch 4 x 131072 tokens,
    top-k 8/32/64 (bf16 O, no LSE), each launch timed with HIP events."""
    cfg = workload.CONFIGS["sweep_128k_b4"]
    N, B = cfg.num_blocks, cfg.batch
    ids = workload.make_ids(cfg, batch=B)
    q, k, v = workload.make_qkv(cfg, batch=B)
    Q, K, V = bf16_dev(q), bf16_dev(k), bf16_dev(v)
    del q, k, v
    d_ids = torch.from_numpy(ids).cuda()
    out = {"workload": "batch 4 x 131072 tokens, 16 blocks x 8192, sink 64, chunk 32, "
                       "Llama-3.1-8B layer shape; every block's Phase-1, bf16 O"}
    rows = []
    star_flops, star_ms = 0, 0.0
    for i in range(N):
        n_s = P.phase1_len(cfg.L, N, i, cfg.sink, cfg.chunk, 0, P.PREFIX_ANCHOR)
        O = torch.empty((B, n_s, cfg.Hq, cfg.d), dtype=torch.bfloat16, device="cuda")
        P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, 0, None, P.PREFIX_ANCHOR,
                      o_dtype=P.OUT_BF16, return_lse=False, out=O)
        t = Timer(spin=True)
        for _ in range(reps):
            with t:
                P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, 0, None, P.PREFIX_ANCHOR,
                              o_dtype=P.OUT_BF16, return_lse=False, out=O)
        torch.cuda.synchronize()
        star_ms += t.mean_ms()
        star_last_ms = t.mean_ms()
        star_flops += B * causal_flops(n_s, cfg.Hq, cfg.d)
        del O
    for topk in (8, 32, 64):
        sel = P.maxidf_summaries(d_ids, N, cfg.chunk, topk, cfg.vocab)
        fl, ms, last = 0, 0.0, None
        for i in range(N):
            n_i = P.phase1_len(cfg.L, N, i, cfg.sink, cfg.chunk, topk)
            O = torch.empty((B, n_i, cfg.Hq, cfg.d), dtype=torch.bfloat16, device="cuda")
            P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, topk, sel, o_dtype=P.OUT_BF16,
                          return_lse=False, out=O)
            t = Timer(spin=True)
            for _ in range(reps):
                with t:
                    P.phase1_attn(Q, K, V, N, i, cfg.sink, cfg.chunk, topk, sel,
                                  o_dtype=P.OUT_BF16, return_lse=False, out=O)
            torch.cuda.synchronize()
            ms += t.mean_ms()
            fl += B * causal_flops(n_i, cfg.Hq, cfg.d)
            last = (n_i, t.mean_ms(), B * causal_flops(n_i, cfg.Hq, cfg.d))
            del O
        n_s = 2 * cfg.Lb
        model_last, model_all = model_ratios(topk, cfg.L, N, cfg.sink, cfg.chunk)
        rows.append({"topk": topk, "sigma": topk * cfg.chunk, "pulsar_ms_all_blocks": ms,
                     "pulsar_tflops": fl / (ms * 1e-3) / 1e12,
                     "flop_ratio_star_over_pulsar_all_blocks": star_flops / fl,
                     "time_ratio_star_over_pulsar_all_blocks": star_ms / ms,
                     "model_ratio_all_blocks": model_all,
                     "last_block_rows": last[0],
                     "last_block_ms": last[1],
                     "flop_ratio_star_over_pulsar_last_block":
                         causal_flops(n_s, cfg.Hq, cfg.d) / causal_flops(last[0], cfg.Hq, cfg.d),
                     "time_ratio_star_over_pulsar_last_block": star_last_ms / last[1],
                     "model_ratio_last_block": model_last})
    out["anchor"] = {"ms_all_blocks": star_ms, "last_block_ms": star_last_ms,
                     "tflops": star_flops / (star_ms * 1e-3) / 1e12}
    out["pulsar"] = rows
    del Q, K, V
    torch.cuda.empty_cache()
    return out, ids


def run_sweep(args):
    out, ids = cfg5_sweep()
    out = {"metric": "anchor vs Pulsar Phase-1 sweep; Max-IDF batch sweep", "config": out}
    cfg = workload.CONFIGS["sweep_128k_b4"]
    N, B = cfg.num_blocks, cfg.batch
    # Max-IDF over batches of 128K sequences: latency-bound at small batch,
    # HBM-bound once the ids no longer fit the caches
    idf_rows = []
    for batch in (1, 8, 64, 256, 512, 1024):
        idsb = np.concatenate([ids] * ((batch + B - 1) // B))[:batch]
        d = torch.from_numpy(np.ascontiguousarray(idsb)).cuda()
        wsb = torch.empty(max(P.maxidf_workspace_bytes(batch, cfg.L, N, cfg.chunk, cfg.vocab), 16),
                          dtype=torch.uint8, device="cuda")
        P.maxidf_summaries(d, N, cfg.chunk, 32, cfg.vocab, workspace=wsb)
        t = Timer(spin=True)
        for _ in range(5):
            with t:
                P.maxidf_summaries(d, N, cfg.chunk, 32, cfg.vocab, workspace=wsb)
        torch.cuda.synchronize()
        ms = t.mean_ms()
        byts = batch * (cfg.L * 4 + N * 32 * 4)
        idf_rows.append({"batch": batch, "ms": ms, "tokens_per_s": batch * cfg.L / (ms * 1e-3),
                         "gbps_algorithmic": byts / (ms * 1e-3) / 1e9,
                         "pct_hbm_peak": 100 * byts / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS})
        del d
    out["maxidf"] = idf_rows
    print(json.dumps(out), flush=True)


class _Null:
    def __enter__(self):
        return self

    def __exit__(self, *exc):
        return False


def _smi_sample():
    """Socket power (W) and per-XCD graphics clocks (MHz) from amd-smi, or None."""
    try:
        out = subprocess.run(["amd-smi", "metric", "--power", "--clock"], capture_output=True,
                             text=True, timeout=10).stdout
    except (OSError, subprocess.SubprocessError):
        return None
    power, clocks, in_gfx = None, [], False
    for line in out.splitlines():
        t = line.strip()
        if t.startswith("SOCKET_POWER:"):
            try:
                power = float(t.split()[1])
            except (IndexError, ValueError):
                pass
        elif t.startswith("GFX_"):
            in_gfx = True
        elif in_gfx and t.startswith("CLK:"):
            try:
                clocks.append(float(t.split()[1]))
            except (IndexError, ValueError):
                pass
            in_gfx = False
        elif t.endswith(":") and not t.startswith("GFX_"):
            in_gfx = False
    return power, clocks


def run_power(args):
    """Phase-1 block 15 (the timed launch) back to back for --power-seconds,
    with the socket power and the graphics clocks sampled once a second."""
    cfg = workload.CONFIGS["llama8b_128k"]
    N, i_last = cfg.num_blocks, cfg.num_blocks - 1
    ids = workload.make_ids(cfg, batch=1)
    q, k, v = workload.make_qkv(cfg, batch=1)
    Q, K, V = bf16_dev(q), bf16_dev(k), bf16_dev(v)
    sel = P.maxidf_summaries(torch.from_numpy(ids).cuda(), N, cfg.chunk, cfg.topk, cfg.vocab)
    n = P.phase1_len(cfg.L, N, i_last, cfg.sink, cfg.chunk, cfg.topk)
    O = torch.empty((1, n, cfg.Hq, cfg.d), dtype=torch.float32, device="cuda")
    launch = lambda: P.phase1_attn(Q, K, V, N, i_last, cfg.sink, cfg.chunk, cfg.topk, sel,
                                   out=O, return_lse=False)
    for _ in range(3):
        launch()
    torch.cuda.synchronize()
    idle = _smi_sample()
    samples, stop = [], threading.Event()

    def sampler():
        while not stop.wait(1.0):
            smp = _smi_sample()
            if smp is not None:
                samples.append(smp)

    th = threading.Thread(target=sampler)
    th.start()
    t0, count = time.time(), 0
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    while time.time() - t0 < args.power_seconds:
        for _ in range(25):
            launch()
        count += 25
        torch.cuda.synchronize()
    e1.record()
    torch.cuda.synchronize()
    stop.set()
    th.join()
    ms = e0.elapsed_time(e1) / count
    busy = [s for s in samples if s[0] is not None]
    print(json.dumps({
        "what": "Phase-1 block 15 (128K workload) back to back; amd-smi samples once a second",
        "launches": count, "ms_per_launch": ms,
        "tflops": causal_flops(n, cfg.Hq, cfg.d) / (ms * 1e-3) / 1e12,
        "idle": None if idle is None else {"socket_power_w": idle[0], "gfx_clk_mhz": idle[1]},
        "busy": [{"socket_power_w": p, "gfx_clk_mhz": c} for p, c in busy],
    }), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--sweep", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="leave the anchor-vs-Pulsar sweep out of the default run")
    ap.add_argument("--profile-step", action="store_true",
                    help="only the warm-up and timed steps (for profiler traces)")
    ap.add_argument("--calibrate", action="store_true",
                    help="append a 1 GiB device copy (counter calibration for rocprofv3 --pmc)")
    ap.add_argument("--power-seconds", type=float, default=0.0,
                    help="only Phase-1 block 15 back to back for this long, sampling power "
                         "and clocks")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library runs on a single GPU and has "
              "no multi-GPU path; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.power_seconds > 0:
        run_power(args)
    elif args.sweep:
        run_sweep(args)
    else:
        run_main(args)


if __name__ == "__main__":
    main()
