"""Parity of pulsar_phase2_query with oracle.attention.query_attention.

New tokens attend, without a mask, to the retained shards and to the
generation shard's appended rows up to themselves (Algorithm 1, Phase 2).
Acceptance as for the other attention outputs: O max-abs 1e-2 and relative
L2 1e-2, LSE max-abs 1e-3.
"""
import math

import numpy as np
import pytest
import torch

import paper_2607_20457_amd as P
from oracle import attention as oatt
from paper_2607_20457_amd import workload
from tests._helpers import check_attention, f64, to_dev_bf16

pytestmark = pytest.mark.gpu


def _run_and_check(q, kg, vg, G, k=None, v=None, what=""):
    d = q.shape[-1]
    scale = 1.0 / math.sqrt(d)
    print(f"phase2_query parity: {what}", flush=True)
    o, lse = P.phase2_query(to_dev_bf16(q), to_dev_bf16(kg), to_dev_bf16(vg), G,
                            None if k is None else to_dev_bf16(k),
                            None if v is None else to_dev_bf16(v))
    Hkv = kg.shape[1]
    Ks = f64(k) if k is not None else np.zeros((0, 0, Hkv, d))
    Vs = f64(v) if v is not None else np.zeros((0, 0, Hkv, d))
    o_ref, lse_ref = oatt.query_attention(f64(q), Ks, Vs, f64(kg), f64(vg), G, scale)
    check_attention(o.cpu().numpy(), lse.cpu().numpy(), o_ref, lse_ref, what)


def test_query_encoding_over_128k_shards():
    # 64 query tokens over the 16 retained shards of 8192 keys (the 128K
    # workload's K/V), then their own rows causally
    cfg = workload.CONFIGS["llama8b_128k"]
    _, k, v = workload.make_qkv(cfg, batch=1)
    Ks = np.ascontiguousarray(k[0].reshape(16, 8192, cfg.Hkv, cfg.d))
    Vs = np.ascontiguousarray(v[0].reshape(16, 8192, cfg.Hkv, cfg.d))
    q = workload.bf16_normal(501, (64, cfg.Hq, cfg.d))
    kg = workload.bf16_normal(502, (64, cfg.Hkv, cfg.d))
    vg = workload.bf16_normal(503, (64, cfg.Hkv, cfg.d))
    _run_and_check(q, kg, vg, 0, Ks, Vs, "query encoding 16 x 8192")


@pytest.mark.parametrize("G", [1, 70, 300])
def test_decode_step(G):
    q = workload.bf16_normal(600 + G, (1, 32, 128))
    kg = workload.bf16_normal(601 + G, (G + 1, 8, 128))
    vg = workload.bf16_normal(602 + G, (G + 1, 8, 128))
    k = workload.bf16_normal(603, (4, 512, 8, 128))
    v = workload.bf16_normal(604, (4, 512, 8, 128))
    _run_and_check(q, kg, vg, G, k, v, f"decode G={G}")


@pytest.mark.parametrize("Hq,Hkv,d,Tq,G,ns,S", [
    (32, 8, 128, 40, 5, 0, 0),       # generation shard only, ragged
    (32, 8, 128, 33, 0, 3, 0),       # empty retained shards
    (4, 1, 64, 100, 17, 2, 300),     # the small layer shape, d 64
    (8, 8, 128, 65, 3, 5, 129),      # one query head per KV head
    (16, 8, 64, 31, 0, 6, 77),       # two query heads per KV head
    (32, 8, 128, 40, 4100, 1, 256),  # generation shard over 4096 rows: attention kernel
    (64, 1, 64, 3, 10, 1, 100),      # 64 heads per KV head: no 32-row tile, attention kernel
    (32, 8, 128, 130, 20, 1, 64),    # 520 query rows per KV head: attention kernel, G > 0
    (64, 8, 64, 13, 7, 2, 90),       # 8 heads per KV head: tiles of 4 tokens, the last of 1
    (32, 1, 64, 5, 3, 1, 50),        # 32 heads per KV head: one token per tile
])
def test_shapes(Hq, Hkv, d, Tq, G, ns, S):
    seed = Hq * 7 + Tq + G
    q = workload.bf16_normal(seed, (Tq, Hq, d))
    kg = workload.bf16_normal(seed + 1, (G + Tq, Hkv, d))
    vg = workload.bf16_normal(seed + 2, (G + Tq, Hkv, d))
    k = workload.bf16_normal(seed + 3, (ns, S, Hkv, d)) if ns else None
    v = workload.bf16_normal(seed + 4, (ns, S, Hkv, d)) if ns else None
    _run_and_check(q, kg, vg, G, k, v, f"Hq={Hq} Hkv={Hkv} d={d} Tq={Tq} G={G} shards={ns}x{S}")


def test_peaked_queries():
    # queries scaled x8: the weights concentrate and |O| is of order 1
    q = workload.bf16_normal(700, (16, 32, 128), scale=8.0)
    kg = workload.bf16_normal(701, (16 + 9, 8, 128))
    vg = workload.bf16_normal(702, (16 + 9, 8, 128))
    k = workload.bf16_normal(703, (8, 1024, 8, 128))
    v = workload.bf16_normal(704, (8, 1024, 8, 128))
    _run_and_check(q, kg, vg, 9, k, v, "peaked")


@pytest.mark.parametrize("Hq,Hkv,d,Tq,G,ns,S", [
    (32, 8, 128, 8, 5, 3, 700),      # 32 packed rows: the decode kernel, causal new rows
    (8, 8, 128, 32, 0, 0, 0),        # one head per KV head, new tokens only
    (16, 8, 64, 16, 600, 2, 300),    # generation shard in three key ranges
    (32, 8, 128, 3, 2000, 4, 512),   # eight generation ranges, the last holding the new rows
    (4, 1, 64, 7, 0, 1, 100),        # one KV head
    (32, 1, 128, 1, 40, 2, 333),     # 32 heads per KV head, one token: a full tile
    (32, 8, 128, 1, 0, 0, 0),        # one token, nothing before it: its own row only
])
def test_few_rows_one_launch(Hq, Hkv, d, Tq, G, ns, S):
    # Tq * Hq / Hkv <= 32: shards and generation shard in one decode launch,
    # token t limited to generation rows up to G + t
    seed = 900 + Hq + Tq + G
    q = workload.bf16_normal(seed, (Tq, Hq, d))
    kg = workload.bf16_normal(seed + 1, (G + Tq, Hkv, d))
    vg = workload.bf16_normal(seed + 2, (G + Tq, Hkv, d))
    k = workload.bf16_normal(seed + 3, (ns, S, Hkv, d)) if ns else None
    v = workload.bf16_normal(seed + 4, (ns, S, Hkv, d)) if ns else None
    _run_and_check(q, kg, vg, G, k, v, f"few rows Hq={Hq} Hkv={Hkv} d={d} Tq={Tq} G={G} "
                   f"shards={ns}x{S}")
