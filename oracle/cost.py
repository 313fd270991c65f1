"""Phase-1 cost model (oracle).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.

Appendix "Block-to-Host Scalability Analysis": block i's Phase-1 input has
n_i = L/B + s_sink + i*sigma rows; a host's cost is the sum of F(n_i) over the
blocks mapped to it, and the critical path is the largest host cost.

Table 4 prices one layer of the 8B model at F(n) = c * n^2 FLOPs.  The paper
does not state c; every FLOP cell of Table 4 is reproduced by c = 10240 =
2 * (Hq + Hkv) * d for 32 query heads, 8 KV heads and d = 128 (reading taken
here; only ratios between methods matter).  For kernel throughput the exact
matrix-core work of causal attention is used instead: 4 * d * Hq FLOPs per
unmasked (query, key) pair (two products of 2 * d FLOPs per pair per head).
"""
from __future__ import annotations


def pulsar_len(L: int, B: int, sink: int, sigma: int, i: int) -> int:
    """n_i = L/B + s_sink + i * sigma (the appendix formula, which Table 4
    applies to the last block)."""
    return L // B + sink + i * sigma


def star_len(L: int, B: int) -> int:
    """Star Attention's Phase-1 input: anchor block plus local block."""
    return 2 * (L // B)


def dense_len(L: int) -> int:
    return L


def table4_flops(n: int, c: int = 10240) -> int:
    """Per-layer Phase-1 FLOPs of an n-row input in Table 4's convention."""
    return c * n * n


def host_costs(lengths, mapping, c: int = 10240):
    """C_h = sum over blocks i with pi(i) = h of F(n_i); returns {h: C_h}."""
    out = {}
    for n_i, h in zip(lengths, mapping):
        out[h] = out.get(h, 0) + table4_flops(n_i, c)
    return out


def critical_path(lengths, mapping, c: int = 10240) -> int:
    return max(host_costs(lengths, mapping, c).values())


def causal_pairs(n: int) -> int:
    """Unmasked (query, key) pairs of index-causal attention over n rows."""
    return n * (n + 1) // 2


def causal_attn_flops(n: int, Hq: int, d: int) -> int:
    """Matrix-core FLOPs of causal attention: 4 * d * Hq per unmasked pair."""
    return 4 * d * Hq * causal_pairs(n)


def full_attn_flops(n_q: int, n_k: int, Hq: int, d: int) -> int:
    """Matrix-core FLOPs of unmasked attention of n_q queries over n_k keys."""
    return 4 * d * Hq * n_q * n_k
