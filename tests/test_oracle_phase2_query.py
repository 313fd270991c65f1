"""Pins of oracle.attention.query_attention (Phase-2 attention of new tokens
over the retained shards plus the designated generation shard).

It is tied to a library routine (PyTorch's fp64 scaled-dot-product attention
with an explicit boolean mask over the concatenated keys), to plain causal
attention when there are no shards, and to the merge of per-part partials
(Appendix "Phase 2 Distributed Softmax Merge": merging partials equals
attention over the concatenated keys).
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A


def _case(seed, H, S, Hkv, d, Hq, G, Tq):
    rng = np.random.default_rng(seed)
    K = rng.standard_normal((H, S, Hkv, d))
    V = rng.standard_normal((H, S, Hkv, d))
    Kg = rng.standard_normal((G + Tq, Hkv, d))
    Vg = rng.standard_normal((G + Tq, Hkv, d))
    q = rng.standard_normal((Tq, Hq, d))
    return q, K, V, Kg, Vg


def _sdpa_reference(q, K, V, Kg, Vg, G, scale):
    Tq, Hq, d = q.shape
    Kc = np.concatenate([K.reshape(-1, *K.shape[2:]), Kg], axis=0)
    Vc = np.concatenate([V.reshape(-1, *V.shape[2:]), Vg], axis=0)
    n_ctx = Kc.shape[0] - Kg.shape[0]
    group = Hq // Kc.shape[1]
    keys = np.arange(Kc.shape[0])
    mask = keys[None, :] <= (n_ctx + G + np.arange(Tq))[:, None]       # [Tq, n_keys]
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]                    # [1, Hq, Tq, d]
    kt = torch.from_numpy(np.repeat(Kc, group, axis=1)).permute(1, 0, 2)[None]
    vt = torch.from_numpy(np.repeat(Vc, group, axis=1)).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=torch.from_numpy(mask),
                                                         scale=scale)
    s = (qt @ kt.transpose(-1, -2)) * scale
    s = s.masked_fill(~torch.from_numpy(mask), -math.inf)
    lse = torch.logsumexp(s, dim=-1)
    return o[0].permute(1, 0, 2).numpy(), lse[0].numpy()


@pytest.mark.parametrize("H,S,G,Tq", [(3, 20, 5, 4), (2, 7, 0, 6), (4, 16, 9, 1), (1, 0, 3, 3)])
def test_matches_masked_sdpa(H, S, G, Tq):
    q, K, V, Kg, Vg = _case(H * 100 + S + G + Tq, H, S, 2, 16, 4, G, Tq)
    sc = 1 / math.sqrt(16)
    o, lse = A.query_attention(q, K, V, Kg, Vg, G, sc)
    o_ref, lse_ref = _sdpa_reference(q, K, V, Kg, Vg, G, sc)
    assert np.allclose(o, o_ref, atol=1e-12)
    assert np.allclose(lse, lse_ref, atol=1e-12)


def test_no_shards_is_causal_attention():
    q, K, V, Kg, Vg = _case(5, 0, 0, 2, 8, 4, 0, 9)
    sc = 0.3
    o, lse = A.query_attention(q, K, V, Kg, Vg, 0, sc)
    o_c, lse_c = A.causal_attention(q, Kg, Vg, sc)
    assert np.allclose(o, o_c, atol=1e-12) and np.allclose(lse, lse_c, atol=1e-12)


@pytest.mark.parametrize("G", [0, 4])
def test_equals_merge_of_parts(G):
    # shards (unmasked), the G earlier appended rows (unmasked), the new
    # tokens' own rows (causal square): merged, they give the direct result
    H, S, Hkv, d, Hq, Tq = 3, 12, 2, 8, 4, 5
    q, K, V, Kg, Vg = _case(40 + G, H, S, Hkv, d, Hq, G, Tq)
    sc = 1 / math.sqrt(d)
    parts = [A.partial_attention(q, K[h], V[h], sc) for h in range(H)]
    if G:
        parts.append(A.partial_attention(q, Kg[:G], Vg[:G], sc))
    parts.append(A.causal_attention(q, Kg[G:], Vg[G:], sc))
    o_m, lse_m = A.lse_merge(np.stack([p[0] for p in parts]), np.stack([p[1] for p in parts]))
    o, lse = A.query_attention(q, K, V, Kg, Vg, G, sc)
    assert np.allclose(o, o_m, atol=1e-12) and np.allclose(lse, lse_m, atol=1e-12)
