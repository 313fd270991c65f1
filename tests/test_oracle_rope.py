"""Pins of the rotary-embedding oracle (sparse global positions).

Each test ties ``oracle.rope`` to something other than its own formula: the
rotation of a unit vector by a known angle (direction of rotation, pairing of
the halves, the frequency exponent), rotations as complex multiplication,
composition of rotations, norm preservation, and the relative-position
property that makes preserved global positions meaningful.
"""
import math

import numpy as np
import pytest

from oracle import assembly, rope


def test_unit_vector_d2_turns_counterclockwise():
    # d = 2, w = 1: (1, 0) at position p is (cos p, sin p); (0, 1) is (-sin p, cos p).
    for p in (0.0, 0.5, 1.0, 3.0, 100.0):
        y = rope.rope(np.array([[[1.0, 0.0]]]), np.array([p]), np.array([1.0]))
        assert np.allclose(y[0, 0], [math.cos(p), math.sin(p)], atol=1e-15)
        y = rope.rope(np.array([[[0.0, 1.0]]]), np.array([p]), np.array([1.0]))
        assert np.allclose(y[0, 0], [-math.sin(p), math.cos(p)], atol=1e-15)


def test_pairs_are_the_two_halves_and_the_exponent():
    # d = 4, base 100: w = (1, 100^(-1/2)) = (1, 0.1).  e_0 moves into
    # components 0 and 2 (pairing i with i + d/2, not 2i with 2i+1); e_1 at
    # position 10 turns by 10 * 0.1 = 1 radian.
    w = rope.inv_freq(4, 100.0)
    assert np.allclose(w, [1.0, 0.1], rtol=0, atol=1e-16)
    y = rope.rope(np.array([[[1.0, 0.0, 0.0, 0.0]]]), np.array([0.7]), w)
    assert np.allclose(y[0, 0], [math.cos(0.7), 0.0, math.sin(0.7), 0.0], atol=1e-15)
    y = rope.rope(np.array([[[0.0, 1.0, 0.0, 0.0]]]), np.array([10.0]), w)
    assert np.allclose(y[0, 0], [0.0, math.cos(1.0), 0.0, math.sin(1.0)], atol=1e-15)


def test_inv_freq_llama_base():
    # base 500000, d = 128: w_0 = 1, w_63 = 500000^(-126/128)
    w = rope.inv_freq(128, 500000.0)
    assert w[0] == 1.0
    assert math.isclose(w[63], 500000.0 ** (-126 / 128), rel_tol=1e-15)
    assert np.all(np.diff(w) < 0)


@pytest.mark.parametrize("seed", range(4))
def test_equals_complex_multiplication(seed):
    rng = np.random.default_rng(seed)
    n, H, d = 9, 3, 16
    x = rng.standard_normal((n, H, d))
    pos = rng.integers(0, 200000, size=n)
    w = rope.inv_freq(d, 10000.0)
    z = (x[..., : d // 2] + 1j * x[..., d // 2:]) * np.exp(1j * pos[:, None, None] * w)
    y = rope.rope(x, pos, w)
    assert np.allclose(y[..., : d // 2], z.real, atol=1e-12)
    assert np.allclose(y[..., d // 2:], z.imag, atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_composition_identity_and_norm(seed):
    rng = np.random.default_rng(100 + seed)
    n, H, d = 7, 2, 32
    x = rng.standard_normal((n, H, d))
    w = rope.inv_freq(d, 1e6)
    p1 = rng.integers(0, 70000, size=n)
    p2 = rng.integers(0, 70000, size=n)
    assert np.allclose(rope.rope(rope.rope(x, p1, w), p2, w), rope.rope(x, p1 + p2, w), atol=1e-9)
    assert np.array_equal(rope.rope(x, np.zeros(n), w), x)
    y = rope.rope(x, p1, w)
    # every pair keeps its length
    assert np.allclose(np.hypot(y[..., : d // 2], y[..., d // 2:]),
                       np.hypot(x[..., : d // 2], x[..., d // 2:]), atol=1e-12)


@pytest.mark.parametrize("seed", range(4))
def test_scores_depend_on_position_differences_only(seed):
    rng = np.random.default_rng(200 + seed)
    d = 64
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, d))
    w = rope.inv_freq(d, 500000.0)
    m, n, c = (int(v) for v in rng.integers(0, 100000, size=3))
    s1 = np.sum(rope.rope(q, np.array([m]), w) * rope.rope(k, np.array([n]), w))
    s2 = np.sum(rope.rope(q, np.array([m + c]), w) * rope.rope(k, np.array([n + c]), w))
    assert math.isclose(s1, s2, rel_tol=1e-9, abs_tol=1e-9)


def test_sparse_positions_are_the_global_rotation_gathered():
    # An assembled input's rows rotated by their global positions are the rows
    # of the whole context rotated by position and then gathered.
    rng = np.random.default_rng(7)
    L, nb, sink, chunk, k, H, d = 256, 4, 8, 8, 2, 2, 16
    x = rng.standard_normal((L, H, d))
    w = rope.inv_freq(d, 10000.0)
    sel = np.stack([np.sort(rng.choice(L // nb // chunk, k, replace=False)) for _ in range(nb)])
    pos = assembly.phase1_positions(L, nb, 3, sink, chunk, k, sel)
    whole = rope.rope(x, np.arange(L), w)
    assert np.array_equal(rope.rope(x[pos], pos, w), whole[pos])


# ------------------------------------------------------------ contiguous mode --
# Appendix "RoPE Position ID Assignment", contiguous: block i's assembled input
# is renumbered 0 .. n_i - 1 and Phase-2 positions start just past the longest
# assembled input.

def test_contiguous_positions_hand_example():
    # L = 64, 4 blocks of 16, sink 2, chunk 2, top-1: block 3's input is
    # [sink 0 1 | Sigma_0 | Sigma_1 | Sigma_2 | B_3] with 2 + 3*2 + 16 = 24 rows
    sel = np.array([[5], [0], [7], [3]])
    sp = rope.phase1_rope_positions(64, 4, 3, 2, 2, 1, sel, pos_mode=rope.SPARSE)
    assert sp.tolist() == [0, 1, 10, 11, 16, 17, 46, 47] + list(range(48, 64))
    ct = rope.phase1_rope_positions(64, 4, 3, 2, 2, 1, sel, pos_mode=rope.CONTIGUOUS)
    assert ct.tolist() == list(range(24))
    # the longest input is block 3's: 24 rows, so queries start at 24
    q = rope.query_positions(64, 4, 2, 2, 1, Tq=3, pos_mode=rope.CONTIGUOUS)
    assert q.tolist() == [24, 25, 26]
    # sparse queries follow the 64-token context; G earlier tokens shift them
    assert rope.query_positions(64, 4, 2, 2, 1, Tq=2, G=5).tolist() == [69, 70]
    assert rope.query_positions(64, 4, 2, 2, 1, Tq=1, G=5,
                                pos_mode=rope.CONTIGUOUS).tolist() == [29]


@pytest.mark.parametrize("mode", [assembly.PREFIX_SUMMARY, assembly.PREFIX_ANCHOR,
                                  assembly.PREFIX_EVEN])
def test_contiguous_block0_equals_sparse_and_queries_come_after_every_row(mode):
    # Input_0 = [B_0] sits at global positions 0 .. Lb-1: both modes agree.
    # Contiguous queries come after every row of every block's input, and the
    # first one directly after the longest input.
    rng = np.random.default_rng(3)
    L, N, s, m, k = 512, 8, 8, 4, 3
    sel = np.stack([np.sort(rng.choice(L // N // m, k, replace=False)) for _ in range(N)])
    a = rope.phase1_rope_positions(L, N, 0, s, m, k, sel, mode, rope.SPARSE)
    b = rope.phase1_rope_positions(L, N, 0, s, m, k, sel, mode, rope.CONTIGUOUS)
    assert np.array_equal(a, b)
    q = rope.query_positions(L, N, s, m, k, Tq=4, prefix_mode=mode, pos_mode=rope.CONTIGUOUS)
    last = max(rope.phase1_rope_positions(L, N, i, s, m, k, sel, mode, rope.CONTIGUOUS).max()
               for i in range(N))
    assert q[0] == last + 1
    if mode == assembly.PREFIX_ANCHOR:
        assert q[0] == 2 * (L // N)          # Star-style [B_0 || B_i], 2 Lb rows


def test_contiguous_keeps_distances_inside_b_i_only():
    # Rotated scores depend on position differences.  Within B_i the rows are
    # consecutive in both modes, so scores between them agree; a summary row
    # is k*m*(i-1-j)+... rows away in contiguous mode but blocks away in
    # sparse mode, so its scores against B_i differ.
    rng = np.random.default_rng(11)
    L, N, s, m, k, H, d = 256, 4, 4, 4, 2, 1, 16
    sel = np.stack([np.sort(rng.choice(L // N // m, k, replace=False)) for _ in range(N)])
    x = rng.standard_normal((L, H, d))
    w = rope.inv_freq(d, 10000.0)
    src = assembly.phase1_positions(L, N, 3, s, m, k, sel)
    sp = rope.assembled_rope(x, src, rope.phase1_rope_positions(L, N, 3, s, m, k, sel), w)
    ct = rope.assembled_rope(x, src, rope.phase1_rope_positions(L, N, 3, s, m, k, sel,
                                                                pos_mode=rope.CONTIGUOUS), w)
    n, Lb = len(src), L // N
    bi = np.arange(n - Lb, n)
    g_sp = np.einsum("rhd,chd->rc", sp[bi], sp[bi])
    g_ct = np.einsum("rhd,chd->rc", ct[bi], ct[bi])
    np.testing.assert_allclose(g_sp, g_ct, atol=1e-9)
    summ = s  # first summary row
    c_sp = np.einsum("rhd,hd->r", sp[bi], sp[summ])
    c_ct = np.einsum("rhd,hd->r", ct[bi], ct[summ])
    assert np.max(np.abs(c_sp - c_ct)) > 1e-3


def test_assembled_rope_turns_each_row_by_its_own_position():
    # d = 2, w = 1: row r of (1, 0) rows, gathered from any positions and
    # rotated contiguously, is (cos r, sin r)
    x = np.zeros((10, 1, 2))
    x[:, 0, 0] = 1.0
    src = np.array([7, 2, 2, 9])
    y = rope.assembled_rope(x, src, np.arange(4), np.array([1.0]))
    for r in range(4):
        assert np.allclose(y[r, 0], [math.cos(r), math.sin(r)], atol=1e-15)
