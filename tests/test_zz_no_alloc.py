"""pulsar_phase2_query_noalloc (partials in the library's static per-device
scratch) against pulsar_phase2_query (caller workspace) through the C ABI:
two calls in a row on one device, the second with a smaller input, each
compared with the workspace call bit for bit and with the fp64 oracle."""
import math

import numpy as np
import pytest
import torch

import paper_2607_20457_amd as P
from oracle import attention
from paper_2607_20457_amd import workload
from tests._helpers import check_attention, f64, gpu_available, to_dev_bf16

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not gpu_available(), reason="needs a GPU")]


def _case(seed, n_shards, S, G, Tq, Hq=32, Hkv=8, d=128):
    q = workload.bf16_normal(seed, (Tq, Hq, d))
    K = workload.bf16_normal(seed + 1, (n_shards, S, Hkv, d))
    V = workload.bf16_normal(seed + 2, (n_shards, S, Hkv, d))
    Kg = workload.bf16_normal(seed + 3, (G + Tq, Hkv, d))
    Vg = workload.bf16_normal(seed + 4, (G + Tq, Hkv, d))
    return q, K, V, Kg, Vg


def _check(q, K, V, Kg, Vg, G, what):
    print(f"no-alloc phase-2 query: {what} q={q.shape} shards={K.shape} G={G}", flush=True)
    dq, dK, dV, dKg, dVg = (to_dev_bf16(x) for x in (q, K, V, Kg, Vg))
    o_s, l_s = P.phase2_query_noalloc(dq, dKg, dVg, G, dK, dV)
    torch.cuda.synchronize()
    o_w, l_w = P.phase2_query(dq, dKg, dVg, G, dK, dV)
    torch.cuda.synchronize()
    assert torch.equal(o_s, o_w), what
    assert torch.equal(l_s, l_w), what
    d = q.shape[-1]
    o_ref, l_ref = attention.query_attention(f64(q), f64(K), f64(V), f64(Kg), f64(Vg), G,
                                             1 / math.sqrt(d))
    check_attention(o_s.cpu().numpy(), l_s.cpu().numpy(), o_ref, l_ref, what)


def test_noalloc_matches_workspace_call_twice_second_smaller():
    # first: the 64-token query encoding over 16 shards of 8192 keys (the
    # benchmark's shape, about 35 MB of partials); then a one-token decode
    # step over 4 shards of 1000 keys after 37 appended rows, which reuses the
    # same scratch with a different partial layout
    big = _case(7001, 16, 8192, 0, 64)
    _check(*big, G=0, what="encoding 64 tokens, 16 x 8192")
    small = _case(7101, 4, 1000, 37, 1)
    _check(*small, G=37, what="decode step, 4 x 1000, G 37")


def test_noalloc_rejects_partials_beyond_the_scratch():
    q, K, V, Kg, Vg = _case(7201, 2, 64, 0, 1)
    dq, dK, dV, dKg, dVg = (to_dev_bf16(x) for x in (q, K, V, Kg, Vg))
    need = P.api._lib.lib().pulsar_phase2_query_workspace_bytes(16, 256, 8192, 0, 32, 8, 128)
    assert need > (64 << 20)
    big_q = torch.zeros((256, 32, 128), dtype=torch.bfloat16, device="cuda")
    big_K = torch.zeros((16, 8192, 8, 128), dtype=torch.bfloat16, device="cuda")
    big_g = torch.zeros((256, 8, 128), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(P.api._lib.PulsarError) as e:
        P.phase2_query_noalloc(big_q, big_g, big_g, 0, big_K, big_K)
    assert e.value.status == -5
    torch.cuda.synchronize()
    # the entry point still works afterwards
    _check(q, K, V, Kg, Vg, G=0, what="after a rejected call")
