"""Parity of pulsar_rope with the fp64 oracle (oracle.rope).

The output is bf16, so the bar is one rounding: every element lies within
half a bf16 ulp of the exact rotation plus the fp32 evaluation error (a few
fp32 ulps of the input pair's size, which matters only where the rotation
cancels to a tiny value).  Positions go up to and past 131072, where the
fp64 angle matters.
"""
import math

import numpy as np
import pytest
import torch

import paper_2607_20457_amd as P
from oracle import assembly
from oracle import rope as orope
from paper_2607_20457_amd import workload
from tests._helpers import f64, to_dev_bf16, to_dev_i32

pytestmark = pytest.mark.gpu


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def check_rounding(got_bits, ref, x, what=""):
    """got = bf16 rounding of an fp32 evaluation of the rotation.  Bound per
    element: half a bf16 ulp of the exact value (slightly widened for the
    rounding of the fp32 value) plus the fp32 evaluation error, a few fp32
    ulps of the input pair's size (it dominates only where the rotation
    cancels to a tiny result)."""
    got = f64(got_bits)
    d = x.shape[-1]
    pair = np.abs(x[..., : d // 2]) + np.abs(x[..., d // 2:])
    pair = np.concatenate([pair, pair], axis=-1)
    mag = np.abs(ref)
    ulp = np.exp2(np.floor(np.log2(np.maximum(mag, 2.0 ** -126))) - 7)
    bound = 0.5 * ulp * (1 + 2.0 ** -7) + 4 * 2.0 ** -24 * pair
    err = np.abs(got - ref)
    worst = np.max(err / bound)
    assert worst <= 1.0, f"{what}: error {worst:.3f} x the rounding bound"
    frac = np.mean(err > 0.5 * ulp + 4 * 2.0 ** -24 * pair)
    assert frac <= 1e-4, f"{what}: {frac:.2e} of the elements not correctly rounded"


def llama3_table(d: int, base: float = 500000.0) -> np.ndarray:
    """A scaled frequency table (the Llama-3.1 scheme: factor 8, 1..4, 8192),
    to exercise the caller-given table; the oracle gets the same fp32 values."""
    w = orope.inv_freq(d, base)
    wl = 2 * math.pi / w
    lo, hi = 8192 / 1.0, 8192 / 4.0
    smooth = (8192 / wl - 1.0) / (4.0 - 1.0)
    scaled = np.where(wl > lo, w / 8.0, np.where(wl < hi, w, (1 - smooth) * w / 8.0 + smooth * w))
    return scaled.astype(np.float32)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("H,n,batch", [(1, 1, 1), (3, 37, 2), (32, 300, 1), (8, 129, 2)])
@pytest.mark.parametrize("posmode", ["rows", "random", "offset"])
def test_rope_matches_oracle(d, H, n, batch, posmode):
    rng = np.random.default_rng(d * 1000 + H * 10 + n)
    x = workload.bf16_normal(int(rng.integers(1 << 30)), (batch, n, H, d))
    pos = None
    off = 0
    if posmode == "rows":
        p64 = np.broadcast_to(np.arange(n), (batch, n))
    elif posmode == "random":
        p64 = rng.integers(0, 1 << 20, size=(batch, n))
        pos = to_dev_i32(p64)
    else:
        off = 131072
        p64 = np.broadcast_to(np.arange(n), (batch, n)) + off
    X = to_dev_bf16(x)
    P.rope_(X, pos, pos_offset=off, base=500000.0)
    ref = orope.rope(f64(x), p64, orope.inv_freq(d, 500000.0))
    check_rounding(_bits(X), ref, f64(x), f"d={d} H={H} n={n} {posmode}")


@pytest.mark.parametrize("d", [64, 128])
def test_rope_caller_table(d):
    x = workload.bf16_normal(77 + d, (2, 200, 4, d))
    table = llama3_table(d)
    rng = np.random.default_rng(3)
    p64 = rng.integers(0, 140000, size=(2, 200))
    X = to_dev_bf16(x)
    P.rope_(X, to_dev_i32(p64), inv_freq=table)
    ref = orope.rope(f64(x), p64, table.astype(np.float64))
    check_rounding(_bits(X), ref, f64(x), f"table d={d}")


def test_rope_128k_queries_sampled():
    # the 128K workload's query tensor (32 heads, d 128), rotated by row
    # position; 512 rows sampled, the first and last included
    cfg = workload.CONFIGS["llama8b_128k"]
    q, _, _ = workload.make_qkv(cfg, batch=1)
    Q = to_dev_bf16(q)
    P.rope_(Q, None, base=500000.0)
    got = _bits(Q)[0]
    rng = np.random.default_rng(11)
    rows = np.unique(np.r_[0, 1, cfg.L - 1, rng.integers(0, cfg.L, 509)])
    ref = orope.rope(f64(q[0, rows]), rows, orope.inv_freq(128, 500000.0))
    check_rounding(got[rows], ref, f64(q[0, rows]), "128K queries")


def test_rope_assembled_rows_equal_gathered_rotation():
    # sparse mode: rows of block 15's input rotated at their global positions
    # are the rotated context rows at those positions, bit for bit
    cfg = workload.CONFIGS["llama8b_128k"]
    ids = workload.make_ids(cfg, batch=1)
    sel = P.maxidf_summaries(to_dev_i32(ids), cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab)
    pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, 15, cfg.sink, cfg.chunk, cfg.topk,
                                    sel.cpu().numpy()[0])
    k = workload.bf16_normal(5, (1, cfg.L, 8, 128))
    K = to_dev_bf16(k)
    Ka = to_dev_bf16(np.ascontiguousarray(k[:, pos]))
    P.rope_(K, None)
    P.rope_(Ka, to_dev_i32(pos[None]))
    assert torch.equal(Ka.view(torch.int16), K[:, torch.from_numpy(pos).cuda()].view(torch.int16))


def test_rope_empty_and_position_zero():
    X = torch.empty((1, 0, 4, 128), dtype=torch.bfloat16, device="cuda")
    P.rope_(X)  # nothing to do
    x = workload.bf16_normal(9, (1, 1, 4, 128))
    X = to_dev_bf16(x)
    P.rope_(X)  # row 0: position 0, the identity
    assert np.array_equal(_bits(X), x.view(np.uint16))


# ------------------------------------------------ assembled inputs, contiguous --

def _gather_case(cfg, i, mode, batch=2, seed=5):
    x = workload.bf16_normal(seed, (batch, cfg.L, cfg.Hkv, cfg.d))
    rng = np.random.default_rng(seed)
    C = cfg.Lb // cfg.chunk
    sel = np.stack([np.stack([np.sort(rng.choice(C, cfg.topk, replace=False))
                              for _ in range(cfg.num_blocks)]) for _ in range(batch)])
    return x, sel.astype(np.int32)


GATHER_CASES = [
    workload.Config("g_tiny", L=4096, vocab=1, num_blocks=4, sink=64, chunk=16, topk=4,
                    Hq=4, Hkv=3, d=64),
    workload.Config("g_ragged", L=4000, vocab=1, num_blocks=4, sink=40, chunk=20, topk=3,
                    Hq=8, Hkv=5, d=128),
    workload.Config("g_128k", L=131072, vocab=1, num_blocks=16, sink=64, chunk=32, topk=32,
                    Hq=32, Hkv=8, d=128),
]


@pytest.mark.parametrize("cfg", GATHER_CASES, ids=lambda c: c.name)
@pytest.mark.parametrize("mode", [P.PREFIX_SUMMARY, P.PREFIX_ANCHOR, P.PREFIX_EVEN])
def test_gather_contiguous_sparse_and_plain(cfg, mode):
    i = cfg.num_blocks - 1
    batch = 1 if cfg.L > 100000 else 2
    x, sel = _gather_case(cfg, i, mode, batch)
    X, S = to_dev_bf16(x), to_dev_i32(sel)
    print(f"gather: {cfg.name} block {i} mode {mode} batch {batch}", flush=True)
    w = orope.inv_freq(cfg.d, 500000.0)
    plain = P.phase1_gather(X, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S, mode,
                            P.POS_NONE)
    sparse = P.phase1_gather(X, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S, mode,
                             P.POS_SPARSE)
    cont = P.phase1_gather(X, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S, mode,
                           P.POS_CONTIGUOUS)
    whole = X.clone()
    P.rope_(whole)                                   # sparse: rotate once, then gather
    torch.cuda.synchronize()
    for b in range(batch):
        sel_b = None if mode != P.PREFIX_SUMMARY else sel[b]
        pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk,
                                        sel_b, mode)
        assert np.array_equal(_bits(plain[b]), x[b][pos])                 # bit-exact gather
        assert np.array_equal(_bits(sparse[b]), _bits(whole[b])[pos])    # same rotation code
        rows = np.unique(np.concatenate([np.arange(min(200, len(pos))),
                                         np.linspace(0, len(pos) - 1, 300).astype(int)]))
        rot = orope.phase1_rope_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk,
                                          cfg.topk, sel_b, mode, orope.CONTIGUOUS)
        xr = f64(x[b][pos[rows]])                    # the sampled rows' inputs
        idx = np.arange(len(rows))
        ref = orope.assembled_rope(xr, idx, rot[rows], w)
        check_rounding(_bits(cont[b])[rows], ref, xr, f"{cfg.name} mode {mode} contiguous")
        ref = orope.assembled_rope(xr, idx, pos[rows], w)
        check_rounding(_bits(sparse[b])[rows], ref, xr, f"{cfg.name} mode {mode} sparse")


def _round_bf16(a):
    """fp64 -> bf16 (nearest-even through fp32), back as fp64."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def test_contiguous_phase1_and_phase2_positions_end_to_end():
    # Contiguous mode (Appendix "RoPE Position ID Assignment"): block i's
    # input renumbered 0..n_i-1, attention over the materialised rows (the
    # identity map), and Phase-2 queries from max_i n_i on.  The oracle rotates
    # in fp64 and rounds the rotated rows to bf16, the precision the
    # materialised rows have.
    from oracle import attention
    cfg = workload.CONFIGS["tiny"]
    q, k, v = workload.make_qkv(cfg)
    ids = workload.make_ids(cfg)
    from oracle import maxidf
    sel, _, _, _ = maxidf.maxidf_summaries(ids, cfg.num_blocks, cfg.chunk, cfg.topk, cfg.vocab)
    Q, K, V, S = to_dev_bf16(q), to_dev_bf16(k), to_dev_bf16(v), to_dev_i32(sel)
    w = orope.inv_freq(cfg.d, 500000.0)
    scale = 1 / math.sqrt(cfg.d)
    for i in (1, cfg.num_blocks - 1):
        args = (cfg.num_blocks, i, cfg.sink, cfg.chunk, cfg.topk, S, P.PREFIX_SUMMARY)
        Qc = P.phase1_gather(Q, *args, P.POS_CONTIGUOUS)
        Kc = P.phase1_gather(K, *args, P.POS_CONTIGUOUS)
        Vc = P.phase1_gather(V, *args, P.POS_NONE)
        n = Qc.shape[1]
        o, lse = P.phase1_attn(Qc, Kc, Vc, 1, 0, 0, cfg.chunk, 0)
        torch.cuda.synchronize()
        pos = assembly.phase1_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk,
                                        cfg.topk, sel[0])
        rot = orope.phase1_rope_positions(cfg.L, cfg.num_blocks, i, cfg.sink, cfg.chunk,
                                          cfg.topk, sel[0], pos_mode=orope.CONTIGUOUS)
        qa = _round_bf16(orope.assembled_rope(f64(q[0]), pos, rot, w))
        ka = _round_bf16(orope.assembled_rope(f64(k[0]), pos, rot, w))
        o_ref, lse_ref = attention.causal_attention(qa, ka, f64(v[0])[pos], scale)
        from tests._helpers import check_attention
        check_attention(o[0].cpu().numpy(), lse[0].cpu().numpy(), o_ref, lse_ref,
                        f"contiguous block {i}")
        assert n == len(pos)
    # Phase-2 tokens start just past the longest assembled input
    Tq = 3
    qpos = orope.query_positions(cfg.L, cfg.num_blocks, cfg.sink, cfg.chunk, cfg.topk, Tq,
                                 G=2, pos_mode=orope.CONTIGUOUS)
    n_max = P.phase1_len(cfg.L, cfg.num_blocks, cfg.num_blocks - 1, cfg.sink, cfg.chunk,
                         cfg.topk)
    xq = workload.bf16_normal(77, (Tq, cfg.Hq, cfg.d))
    Xq = to_dev_bf16(xq)
    P.rope_(Xq, None, pos_offset=n_max + 2)
    torch.cuda.synchronize()
    ref = orope.rope(f64(xq), qpos, w)
    check_rounding(_bits(Xq), ref, f64(xq), "contiguous Phase-2 queries")
