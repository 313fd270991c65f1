"""GPU parity of Phase-2 partial attention and the online-softmax merge
against the fp64 oracle, and merged partials against dense attention."""
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


def _shards(H, S, Hkv, d, seed):
    k = workload.bf16_normal(seed, (H, S, Hkv, d))
    v = workload.bf16_normal(seed + 1, (H, S, Hkv, d))
    return k, v


def test_phase2_128k_partials_merge_and_dense():
    cfg = workload.CONFIGS["phase2_128k"]
    H, S, Tq = 16, cfg.Lb, 64
    print(f"phase2 parity: shards={H} S={S} Tq={Tq}", flush=True)
    q = workload.bf16_normal(cfg.seed * 10 + 1, (Tq, cfg.Hq, cfg.d))
    k, v = _shards(H, S, cfg.Hkv, cfg.d, cfg.seed * 10 + 2)
    scale = 1 / math.sqrt(cfg.d)
    dq, dk, dv = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v)
    o_parts, lse_parts = P.phase2_partial(dq, dk, dv)
    o, lse = P.lse_merge(o_parts, lse_parts)
    od, lsed = P.phase2_partial(dq, dk.reshape(1, H * S, cfg.Hkv, cfg.d),
                                dv.reshape(1, H * S, cfg.Hkv, cfg.d))
    torch.cuda.synchronize()
    qf, kf, vf = f64(q), f64(k), f64(v)
    refs = [attention.partial_attention(qf, kf[h], vf[h], scale) for h in range(H)]
    for h in range(H):
        check_attention(o_parts[h].cpu().numpy(), lse_parts[h].cpu().numpy(), *refs[h],
                        f"shard {h}")
    o_m, lse_m = attention.lse_merge(np.stack([r[0] for r in refs]), np.stack([r[1] for r in refs]))
    o_dense, lse_dense = attention.dense_attention(qf, kf.reshape(-1, cfg.Hkv, cfg.d),
                                                   vf.reshape(-1, cfg.Hkv, cfg.d), scale)
    check_attention(o.cpu().numpy(), lse.cpu().numpy(), o_m, lse_m, "merged")
    check_attention(o.cpu().numpy(), lse.cpu().numpy(), o_dense, lse_dense, "merged vs dense")
    check_attention(od[0].cpu().numpy(), lsed[0].cpu().numpy(), o_dense, lse_dense, "dense")


@pytest.mark.parametrize("Tq,S,Hq,Hkv,d", [(1, 1024, 4, 1, 64), (5, 1000, 8, 2, 128),
                                            (70, 333, 32, 8, 128), (3, 64, 4, 4, 64)])
def test_phase2_ragged_shapes(Tq, S, Hq, Hkv, d):
    H = 3
    q = workload.bf16_normal(7 + Tq, (Tq, Hq, d))
    k, v = _shards(H, S, Hkv, d, 9 + S)
    o_parts, lse_parts = P.phase2_partial(to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v))
    torch.cuda.synchronize()
    for h in range(H):
        ref = attention.partial_attention(f64(q), f64(k[h]), f64(v[h]), 1 / math.sqrt(d))
        check_attention(o_parts[h].cpu().numpy(), lse_parts[h].cpu().numpy(), *ref, f"shard {h}")


def test_empty_shard_and_missing_partial():
    Tq, Hq, Hkv, d = 4, 8, 2, 64
    q = to_dev_bf16(workload.bf16_normal(1, (Tq, Hq, d)))
    k = torch.empty((2, 0, Hkv, d), dtype=torch.bfloat16, device="cuda")
    o, lse = P.phase2_partial(q, k, k.clone())
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(torch.isneginf(lse))
    # a missing shard (lse = -inf, o = 0) leaves the merge of the rest unchanged
    rng = np.random.default_rng(2)
    op = rng.standard_normal((3, Tq, Hq, d)).astype(np.float32)
    lp = rng.standard_normal((3, Hq, Tq)).astype(np.float32)
    lp[1] = -np.inf
    op[1] = 0
    o3, l3 = P.lse_merge(torch.from_numpy(op).cuda(), torch.from_numpy(lp).cuda())
    o2, l2 = P.lse_merge(torch.from_numpy(op[[0, 2]]).cuda(), torch.from_numpy(lp[[0, 2]]).cuda())
    ref_o, ref_l = attention.lse_merge(op[[0, 2]], lp[[0, 2]])
    torch.cuda.synchronize()
    np.testing.assert_allclose(o3.cpu().numpy(), ref_o, atol=1e-5)
    np.testing.assert_allclose(l3.cpu().numpy(), ref_l, atol=1e-5)
    assert torch.allclose(o3, o2) and torch.allclose(l3, l2)
    # every partial missing: lse -inf, o 0
    o0, l0 = P.lse_merge(torch.zeros((2, Tq, Hq, d), device="cuda"),
                         torch.full((2, Hq, Tq), -math.inf, device="cuda"))
    assert torch.all(o0 == 0) and torch.all(torch.isneginf(l0))


def test_merge_large_gaps():
    rng = np.random.default_rng(5)
    op = rng.standard_normal((4, 2, 4, 8)).astype(np.float32)
    lp = (rng.standard_normal((4, 4, 2)) * 300).astype(np.float32)
    o, lse = P.lse_merge(torch.from_numpy(op).cuda(), torch.from_numpy(lp).cuda())
    ref_o, ref_l = attention.lse_merge(op, lp)
    torch.cuda.synchronize()
    np.testing.assert_allclose(o.cpu().numpy(), ref_o, atol=1e-5)
    np.testing.assert_allclose(lse.cpu().numpy(), ref_l, atol=1e-4)


def test_tiny_phase2_one_query_over_four_shards():
    cfg = workload.CONFIGS["tiny"]
    q_all, k_all, v_all = workload.make_qkv(cfg)
    q = q_all[0, -1:]                                   # one query token
    k = k_all[0].reshape(4, cfg.Lb, cfg.Hkv, cfg.d)     # the four retained shards
    v = v_all[0].reshape(4, cfg.Lb, cfg.Hkv, cfg.d)
    o_parts, lse_parts = P.phase2_partial(to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v))
    o, lse = P.lse_merge(o_parts, lse_parts)
    torch.cuda.synchronize()
    ref = attention.dense_attention(f64(q), f64(k_all[0]), f64(v_all[0]), 1 / math.sqrt(cfg.d))
    check_attention(o.cpu().numpy(), lse.cpu().numpy(), *ref, "tiny phase 2")


def test_phase2_far_larger_later_score():
    Tq, Hq, Hkv, d, S = 8, 8, 2, 128, 700
    q = workload.bf16_bits_to_f32(workload.bf16_normal(3, (Tq, Hq, d))) + 1.0
    kf = workload.bf16_bits_to_f32(workload.bf16_normal(4, (2, S, Hkv, d)))
    kf[1, 300] = 8.0
    qb, kb = workload.f32_to_bf16_bits(q), workload.f32_to_bf16_bits(kf)
    vb = workload.bf16_normal(5, (2, S, Hkv, d))
    o_parts, lse_parts = P.phase2_partial(to_dev_bf16(qb), to_dev_bf16(kb), to_dev_bf16(vb))
    torch.cuda.synchronize()
    for h in range(2):
        ref = attention.partial_attention(f64(qb), f64(kb[h]), f64(vb[h]), 1 / math.sqrt(d))
        check_attention(o_parts[h].cpu().numpy(), lse_parts[h].cpu().numpy(), *ref, f"shard {h}")


@pytest.mark.parametrize("Tq,H,S,Hq,Hkv,d", [
    (1, 2, 1, 32, 8, 128),      # one key
    (1, 3, 31, 32, 8, 128),     # one partial step
    (2, 2, 33, 16, 8, 64),      # group 2, a step and one key
    (4, 5, 1000, 32, 4, 128),   # group 8: 32 packed rows
    (8, 1, 4100, 8, 2, 64),     # group 4, 32 packed rows, many key ranges
    (3, 4, 777, 8, 8, 128),     # group 1
])
def test_decode_kernel_shapes(Tq, H, S, Hq, Hkv, d):
    # few query rows per KV head (Tq * Hq / Hkv <= 32): the decode kernel,
    # one key range per wave, merged per shard
    print(f"decode parity: Tq={Tq} shards={H} S={S} Hq={Hq} Hkv={Hkv} d={d}", flush=True)
    q = workload.bf16_normal(40 + Tq + S, (Tq, Hq, d))
    k, v = _shards(H, S, Hkv, d, 41 + S)
    o_parts, lse_parts = P.phase2_partial(to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v))
    torch.cuda.synchronize()
    for h in range(H):
        ref = attention.partial_attention(f64(q), f64(k[h]), f64(v[h]), 1 / math.sqrt(d))
        check_attention(o_parts[h].cpu().numpy(), lse_parts[h].cpu().numpy(), *ref, f"shard {h}")


def test_decode_step_over_128k_shards_matches_dense():
    # one new token over the 16 retained shards of 8192 keys (the decode
    # step's shard partials), merged, against dense attention over 131072 keys
    cfg = workload.CONFIGS["phase2_128k"]
    H, S = 16, cfg.Lb
    q = workload.bf16_normal(cfg.seed * 10 + 5, (1, cfg.Hq, cfg.d))
    k, v = _shards(H, S, cfg.Hkv, cfg.d, cfg.seed * 10 + 2)
    o_parts, lse_parts = P.phase2_partial(to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v))
    o, lse = P.lse_merge(o_parts, lse_parts)
    torch.cuda.synchronize()
    ref = attention.dense_attention(f64(q), f64(k).reshape(-1, cfg.Hkv, cfg.d),
                                    f64(v).reshape(-1, cfg.Hkv, cfg.d), 1 / math.sqrt(cfg.d))
    check_attention(o.cpu().numpy(), lse.cpu().numpy(), *ref, "decode over 128K")


@pytest.mark.parametrize("H,Tq,Hq,d", [(8, 1, 32, 128), (258, 1, 32, 128), (70, 2, 8, 64)])
def test_merge_many_parts_few_outputs(H, Tq, Hq, d):
    # many partials, few outputs: the merge takes one wavefront per output
    # group, its lanes over the parts; missing parts and large gaps included
    rng = np.random.default_rng(H + Tq)
    op = rng.standard_normal((H, Tq, Hq, d)).astype(np.float32)
    lp = (rng.standard_normal((H, Hq, Tq)) * 30).astype(np.float32)
    lp[::5] = -np.inf
    op[::5] = 0
    lp[:, 0, 0] = -np.inf  # one output with every part missing
    op[:, 0, 0] = 0
    o, lse = P.lse_merge(torch.from_numpy(op).cuda(), torch.from_numpy(lp).cuda())
    torch.cuda.synchronize()
    ref_o, ref_l = attention.lse_merge(op, lp)
    np.testing.assert_allclose(o.cpu().numpy(), ref_o, atol=1e-5, rtol=1e-5)
    np.testing.assert_allclose(lse.cpu().numpy(), ref_l, atol=1e-4, rtol=1e-6)
    assert np.all(o.cpu().numpy()[0, 0] == 0) and np.isneginf(lse.cpu().numpy()[0, 0])
