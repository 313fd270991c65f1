"""Softmax attention, Phase-2 partials and the online-softmax merge (oracle).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.

All arithmetic is fp64 on inputs that are already bf16-rounded.  Library
matrix products are used as single steps; nothing is blocked or fused beyond
cutting the query rows into independent tiles.

* Eq. 1: Attention(Q, K, V) = softmax(Q K^T / sqrt(d)) V, row by row; the
  log-sum-exp of a row is ln sum_c exp(q . k_c / sqrt(d)).
* Phase 1 (Algorithm 1, forward pass over Input_i): every row of the assembled
  input is a query row and attends to the rows at or before it in assembled
  order (index-causal mask).
* Grouped-query attention for the 32-query / 8-KV-head layer (Appendix
  "Hyperparameter Configuration"): query head h reads KV head h // (Hq / Hkv).
* Phase 2 (Algorithm 1; Appendix "Phase 2 Distributed Softmax Merge"): each
  shard h gives (o_h, l_h) over its keys with no mask; the partials are folded
  in shard order with Eq. lse-merge and Eq. out-merge, which equals dense
  attention over the concatenated shards.

Readings taken: scale 1/sqrt(d) with no soft-capping; an empty shard gives
lse = -inf and o = 0 and is skipped by the merge; the merge starts from
shard 0 and evaluates Eq. lse-merge in the form that does not overflow
(identical in exact arithmetic).
"""
from __future__ import annotations

import math

import numpy as np


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def causal_attention(q, k, v, scale: float, row_tile: int = 512):
    """Index-causal attention.  q [n, Hq, d], k/v [n, Hkv, d] -> (o [n, Hq, d],
    lse [Hq, n]) in fp64."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, Hq, d = q.shape
    Hkv = k.shape[1]
    group = Hq // Hkv
    o = np.zeros((n, Hq, d))
    lse = np.zeros((Hq, n))
    for h in range(Hq):
        g = h // group
        for r0 in range(0, n, row_tile):
            r1 = min(n, r0 + row_tile)
            s = (q[r0:r1, h] @ k[:r1, g].T) * scale
            rows = np.arange(r0, r1)[:, None]
            cols = np.arange(r1)[None, :]
            s[cols > rows] = -np.inf
            mx = s.max(axis=1, keepdims=True)
            p = np.exp(s - mx)
            den = p.sum(axis=1, keepdims=True)
            o[r0:r1, h] = (p @ v[:r1, g]) / den
            lse[h, r0:r1] = (mx + np.log(den))[:, 0]
    return o, lse


def causal_attention_rows(q, k, v, scale: float, rows):
    """The same as ``causal_attention`` for the listed rows only."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    n, Hq, d = q.shape
    group = Hq // k.shape[1]
    rows = np.asarray(rows, dtype=np.int64)
    o = np.zeros((rows.size, Hq, d))
    lse = np.zeros((Hq, rows.size))
    for idx, r in enumerate(rows):
        for h in range(Hq):
            g = h // group
            s = (k[:r + 1, g] @ q[r, h]) * scale
            mx = s.max()
            p = np.exp(s - mx)
            den = p.sum()
            o[idx, h] = (p @ v[:r + 1, g]) / den
            lse[h, idx] = mx + math.log(den)
    return o, lse


def gather_rows(x, pos):
    """Rows of a ``[L, H, d]`` per-position tensor at the given global positions."""
    return _f64(x)[np.asarray(pos, dtype=np.int64)]


def phase1_attention(Q, K, V, pos, scale: float, rows=None):
    """Phase-1 attention for one sequence over the assembled input whose rows
    copy the global positions ``pos``.  Q [L, Hq, d], K/V [L, Hkv, d].
    With ``rows`` only those assembled rows are computed (and only the rows
    they can see are gathered)."""
    pos = np.asarray(pos, dtype=np.int64)
    if rows is None:
        q, k, v = gather_rows(Q, pos), gather_rows(K, pos), gather_rows(V, pos)
        return causal_attention(q, k, v, scale)
    rows = np.asarray(rows, dtype=np.int64)
    last = int(rows.max()) + 1
    k, v = gather_rows(K, pos[:last]), gather_rows(V, pos[:last])
    q = np.zeros((last,) + np.shape(Q)[1:])
    q[rows] = gather_rows(Q, pos[rows])
    return causal_attention_rows(q, k, v, scale, rows)


def partial_attention(q, K, V, scale: float):
    """Unmasked attention of q [Tq, Hq, d] over one shard K/V [S, Hkv, d]:
    (o [Tq, Hq, d], lse [Hq, Tq]).  An empty shard gives lse -inf, o 0."""
    q, K, V = _f64(q), _f64(K), _f64(V)
    Tq, Hq, d = q.shape
    S, Hkv = K.shape[0], K.shape[1]
    group = Hq // Hkv
    o = np.zeros((Tq, Hq, d))
    lse = np.full((Hq, Tq), -np.inf)
    if S == 0:
        return o, lse
    for h in range(Hq):
        g = h // group
        s = (q[:, h] @ K[:, g].T) * scale                       # [Tq, S]
        mx = s.max(axis=1, keepdims=True)
        p = np.exp(s - mx)
        den = p.sum(axis=1, keepdims=True)
        o[:, h] = (p @ V[:, g]) / den
        lse[h] = (mx + np.log(den))[:, 0]
    return o, lse


def lse_merge(o_parts, lse_parts):
    """Fold H partials o_parts [H, Tq, Hq, d], lse_parts [H, Hq, Tq] in shard
    order with Eq. lse-merge / Eq. out-merge."""
    o_parts, lse_parts = _f64(o_parts), _f64(lse_parts)
    H = o_parts.shape[0]
    ell = lse_parts[0].T.copy()                                 # [Tq, Hq]
    o = o_parts[0].copy()                                       # [Tq, Hq, d]
    for h in range(1, H):
        ell_h = lse_parts[h].T
        new = np.empty_like(ell)
        for idx in np.ndindex(ell.shape):
            a, b = ell[idx], ell_h[idx]
            if b == -np.inf:                                    # empty shard
                new[idx] = a
            elif a == -np.inf:
                new[idx] = b
            elif b <= a:
                new[idx] = a + math.log1p(math.exp(b - a))
            else:
                new[idx] = b + math.log1p(math.exp(a - b))
        w_old = np.where(ell == -np.inf, 0.0, np.exp(ell - new))
        w_new = np.where(ell_h == -np.inf, 0.0, np.exp(ell_h - new))
        o = w_old[..., None] * o + w_new[..., None] * o_parts[h]
        ell = new
    return o, ell.T.copy()


def dense_attention(q, K, V, scale: float):
    """Unmasked attention over all keys at once (the Phase-2 reference)."""
    return partial_attention(q, K, V, scale)


def query_attention(q, K_shards, V_shards, Kg, Vg, G: int, scale: float):
    """Phase-2 attention of Tq new tokens (Algorithm 1, Phase 2).

    The retained shards K_shards/V_shards [H, S, Hkv, d] are all visible; the
    designated generation shard's appended rows Kg/Vg [G + Tq, Hkv, d] hold G
    earlier query/generated tokens, then the Tq new ones, and new token t sees
    appended rows 0 .. G + t (itself included).  Each token's softmax is taken
    over exactly the keys it sees, concatenated: (o [Tq, Hq, d], lse [Hq, Tq]).

    Reading: Algorithm 1 appends every query and generated token's KV to one
    designated shard; a token sees the tokens before it and itself there."""
    q = _f64(q)
    Kc = np.concatenate([_f64(K_shards).reshape(-1, *K_shards.shape[2:]), _f64(Kg)], axis=0)
    Vc = np.concatenate([_f64(V_shards).reshape(-1, *V_shards.shape[2:]), _f64(Vg)], axis=0)
    n_ctx = Kc.shape[0] - Kg.shape[0]
    Tq, Hq, d = q.shape
    group = Hq // Kc.shape[1]
    # key c is visible to token t iff c <= n_ctx + G + t
    visible = np.arange(Kc.shape[0])[None, :] <= (n_ctx + G + np.arange(Tq))[:, None]
    o = np.zeros((Tq, Hq, d))
    lse = np.zeros((Hq, Tq))
    for h in range(Hq):
        g = h // group
        s = np.where(visible, (q[:, h] @ Kc[:, g].T) * scale, -np.inf)   # [Tq, n_keys]
        mx = s.max(axis=1, keepdims=True)
        p = np.exp(s - mx)
        den = p.sum(axis=1, keepdims=True)
        o[:, h] = (p @ Vc[:, g]) / den
        lse[h] = (mx + np.log(den))[:, 0]
    return o, lse
