"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before any GPU call (runs without a GPU)."""
import ctypes
import os
import re

import pytest

from oracle import assembly
from paper_2607_20457_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pulsar.h")

EINVAL, EUNSUP, EWS = -1, -2, -4
FAKE = 1 << 20  # a non-NULL, 16-byte aligned address that is never dereferenced


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pulsar_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("pulsar_maxidf_summaries", "pulsar_phase1_attn", "pulsar_phase2_partial",
              "pulsar_lse_merge"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = _lib.lib()
    names = declared_functions()
    assert set(names) == set(_lib.SIGNATURES), "binding and header disagree"
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    lib = _lib.lib()
    assert lib.pulsar_version() >= 1
    for code in (0, -1, -2, -3, -4, 7):
        assert isinstance(_lib.status_string(code), str)


@pytest.mark.parametrize("L,N,i,s,m,k,mode", [
    (4096, 4, 3, 64, 16, 4, 0), (32768, 8, 7, 64, 32, 16, 0), (131072, 16, 15, 64, 32, 32, 0),
    (131072, 16, 15, 64, 32, 32, 1), (131072, 16, 0, 64, 32, 32, 0), (1024, 4, 2, 0, 8, 0, 0),
    (1024, 4, 3, 256, 8, 32, 0), (131072, 16, 15, 64, 32, 32, 2), (1000, 4, 3, 7, 5, 3, 2)])
def test_phase1_len_matches_oracle(L, N, i, s, m, k, mode):
    got = _lib.lib().pulsar_phase1_len(L, N, i, s, m, k, mode)
    assert got == assembly.phase1_len(L, N, i, s, m, k, mode)


@pytest.mark.parametrize("args", [
    (4097, 4, 0, 0, 16, 1, 0),      # L % N
    (4096, 4, 4, 0, 16, 1, 0),      # block index out of range
    (4096, 4, 1, 2000, 16, 1, 0),   # sink > Lb
    (4096, 4, 1, 64, 16, 65, 0),    # k * m > Lb
    (4096, 4, 1, 64, 0, 1, 0),      # chunk 0
    (4096, 4, 1, 64, 16, 1, 7),     # mode
    (4096, 4, 1, 64, 16, 1, 3),     # mode
    (4096, 0, 0, 0, 16, 1, 0),      # no blocks
])
def test_phase1_len_rejects(args):
    assert _lib.lib().pulsar_phase1_len(*args) == EINVAL


def test_maxidf_validation():
    f = _lib.lib().pulsar_maxidf_summaries
    ok = dict(ids=FAKE, batch=1, L=4096, N=4, m=16, k=4, V=32000, sel=FAKE)
    def call(**kw):
        a = {**ok, **kw}
        return f(a["ids"], a["batch"], a["L"], a["N"], a["m"], a["k"], a["V"], a["sel"], None,
                 None, a.get("ws"), a.get("wsb", 0), None)
    assert call(L=4100) == EINVAL
    assert call(m=24) == EINVAL          # Lb % m
    assert call(k=65) == EINVAL          # k > chunks per block
    assert call(k=-1) == EINVAL
    assert call(ids=None) == EINVAL
    assert call(ids=FAKE + 4) == EINVAL  # misaligned
    assert call(sel=None) == EINVAL
    assert call(V=0) == EINVAL
    assert call(batch=-1) == EINVAL
    assert call(N=256, L=256 * 64) == EUNSUP
    assert call(m=2) == EUNSUP
    assert call(m=512, L=4 * 1024, k=1) == EUNSUP
    assert call(V=400000) == EUNSUP      # df table beyond one CU's LDS
    assert call(batch=0) == 0            # nothing to do
    need = _lib.lib().pulsar_maxidf_workspace_bytes(1, 4096, 4, 16, 32000)
    assert need > 0
    assert call(ws=FAKE, wsb=need - 1) == EWS
    assert call(ws=FAKE + 8, wsb=need) == EWS   # misaligned


@pytest.mark.parametrize("L,N,V", [(0, 4, 16), (0, 16, 32000), (0, 1, 128256)])
def test_maxidf_empty_context_launches_nothing(L, N, V):
    # A context of no tokens has no chunks (so k must be 0) and nothing to
    # read: with NULL ids and outputs the call returns OK on the host without
    # a launch.  (Before, maxidf_plan picked the register-resident kernel with
    # zero rounds, which read 8192 ids per sequence from the NULL pointer.)
    f = _lib.lib().pulsar_maxidf_summaries
    for batch in (1, 3, 300):
        assert f(None, batch, L, N, 16, 0, V, None, None, None, None, 0, None) == 0
    assert f(None, 1, L, N, 16, 1, V, None, None, None, None, 0, None) == EINVAL  # k > 0


def test_attention_validation():
    f = _lib.lib().pulsar_phase1_attn
    base = [FAKE, FAKE, FAKE, 1, 4096, 4, 1, 64, 4, 1, 64, 16, 4, FAKE, 0, 0.125,
            FAKE, 0, None, None, None, None]
    def call(**kw):
        a = list(base)
        for idx, val in kw.items():
            a[int(idx[1:])] = val
        return f(*a)
    assert call(a4=4097) == EINVAL             # L
    assert call(a5=6, a6=4) == EINVAL          # Hq % Hkv
    assert call(a7=96) == EUNSUP               # head_dim
    assert call(a5=12, a6=4) == EUNSUP         # group 3
    assert call(a13=None) == EINVAL            # selection needed for block 1
    assert call(a15=0.0) == EINVAL             # scale
    assert call(a15=float("inf")) == EINVAL
    assert call(a17=3) == EINVAL               # out dtype
    assert call(a19=FAKE) == EINVAL            # K_keep without V_keep
    assert call(a0=None) == EINVAL
    assert call(a16=FAKE + 2) == EINVAL        # misaligned O
    assert call(a3=0) == 0                     # empty batch


def test_phase2_and_merge_validation():
    lib = _lib.lib()
    p = lib.pulsar_phase2_partial
    assert p(FAKE, FAKE, FAKE, 16, 64, 8192, 32, 7, 128, 0.1, FAKE, FAKE, None, 0, None) == EINVAL
    assert p(FAKE, FAKE, FAKE, 16, 64, 8192, 32, 8, 80, 0.1, FAKE, FAKE, None, 0, None) == EUNSUP
    need = lib.pulsar_phase2_workspace_bytes(16, 64, 8192, 32, 8, 128)
    assert need > 0
    assert p(FAKE, FAKE, FAKE, 16, 64, 8192, 32, 8, 128, 0.1, FAKE, FAKE, None, 0, None) == EWS
    assert p(FAKE, FAKE, FAKE, 16, 64, 8192, 32, 8, 128, 0.1, FAKE, FAKE, FAKE, need - 1,
             None) == EWS
    assert p(None, FAKE, FAKE, 16, 64, 8192, 32, 8, 128, 0.1, FAKE, FAKE, FAKE, need,
             None) == EINVAL
    assert p(FAKE, FAKE, FAKE, 0, 64, 8192, 32, 8, 128, 0.1, FAKE, FAKE, None, 0, None) == 0
    m = lib.pulsar_lse_merge
    assert m(FAKE, FAKE, 0, 64, 32, 128, FAKE, FAKE, None) == EINVAL
    assert m(FAKE, FAKE, 2, 64, 32, 6, FAKE, FAKE, None) == EINVAL
    assert m(None, FAKE, 2, 64, 32, 128, FAKE, FAKE, None) == EINVAL
    assert m(FAKE, FAKE, 2, 0, 32, 128, FAKE, FAKE, None) == 0


def test_binding_refuses_missing_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_lib", None)
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError):
        _lib.lib()


def test_rope_validation():
    f = _lib.lib().pulsar_rope
    table = (ctypes.c_float * 64)(*([1.0] * 64))
    def call(X=FAKE, batch=1, n=4, H=2, d=128, pos=None, off=0, tab=None, base=500000.0):
        return f(X, batch, n, H, d, pos, off, tab, base, None)
    assert call(batch=-1) == EINVAL
    assert call(n=-1) == EINVAL
    assert call(d=63) == EINVAL
    assert call(d=32) == EUNSUP
    assert call(X=None) == EINVAL
    assert call(X=FAKE + 8) == EINVAL      # misaligned
    assert call(base=0.0) == EINVAL
    assert call(base=float("inf")) == EINVAL
    bad = (ctypes.c_float * 64)(*([1.0] * 63 + [float("nan")]))
    assert call(tab=ctypes.cast(bad, ctypes.c_void_p)) == EINVAL
    assert call(n=0) == 0 and call(X=None, batch=0) == 0   # nothing to do
    del table


def test_phase2_query_validation():
    lib = _lib.lib()
    f = lib.pulsar_phase2_query
    ws_need = lib.pulsar_phase2_query_workspace_bytes(4, 8, 1024, 3, 32, 8, 128)
    assert ws_need > 0
    def call(q=FAKE, kg=FAKE, vg=FAKE, G=3, K=FAKE, V=FAKE, ns=4, Tq=8, S=1024, Hq=32, Hkv=8,
             d=128, scale=0.088, o=FAKE, ws=FAKE, wsb=None):
        return f(q, kg, vg, G, K, V, ns, Tq, S, Hq, Hkv, d, scale, o, None, ws,
                 ws_need if wsb is None else wsb, None)
    assert call(G=-1) == EINVAL
    assert call(Hq=30) == EINVAL           # Hq % Hkv
    assert call(scale=0.0) == EINVAL
    assert call(kg=None) == EINVAL
    assert call(o=None) == EINVAL
    assert call(q=FAKE + 4) == EINVAL      # misaligned
    assert call(d=96) == EUNSUP
    assert call(S=1 << 21) == EUNSUP       # a shard past 2 GiB of K
    assert call(ws=None) == EWS
    assert call(wsb=ws_need - 1) == EWS
    assert call(Tq=0) == 0
    # no retained shards but a nonzero shard length: sized without dividing by zero
    assert lib.pulsar_phase2_query_workspace_bytes(0, 1, 512, 3, 32, 8, 128) > 0
    assert lib.pulsar_phase2_workspace_bytes(0, 1, 512, 32, 8, 128) == 0


def test_phase2_query_noalloc_validation():
    # Host-side checks come before any device call: bad arguments, no work
    # and partials beyond the static scratch all return without touching a GPU.
    lib = _lib.lib()
    f = lib.pulsar_phase2_query_noalloc
    def call(q=FAKE, kg=FAKE, vg=FAKE, G=3, K=FAKE, V=FAKE, ns=4, Tq=8, S=1024, Hq=32, Hkv=8,
             d=128, scale=0.088, o=FAKE):
        return f(q, kg, vg, G, K, V, ns, Tq, S, Hq, Hkv, d, scale, o, None, None)
    assert call(G=-1) == EINVAL
    assert call(Hq=30) == EINVAL
    assert call(scale=float("nan")) == EINVAL
    assert call(kg=None) == EINVAL
    assert call(o=FAKE + 4) == EINVAL
    assert call(d=96) == EUNSUP
    assert call(Tq=0) == 0
    ETOOLARGE = -5
    limit = 64 << 20
    big = dict(ns=16, Tq=256, S=8192, G=0)
    assert lib.pulsar_phase2_query_workspace_bytes(16, 256, 8192, 0, 32, 8, 128) > limit
    assert call(**big) == ETOOLARGE
    assert "scratch" in _lib.status_string(ETOOLARGE)
    # the benchmark's 64-token query encoding over 16 shards fits
    assert lib.pulsar_phase2_query_workspace_bytes(16, 64, 8192, 0, 32, 8, 128) <= limit


def test_phase1_positions_validation():
    f = _lib.lib().pulsar_phase1_positions
    def call(sel=FAKE, batch=1, L=4096, N=4, i=2, s=16, m=16, k=4, mode=0, pos=FAKE):
        return f(sel, batch, L, N, i, s, m, k, mode, pos, None)
    assert call(L=4097) == EINVAL                    # L % N
    assert call(i=4) == EINVAL and call(i=-1) == EINVAL
    assert call(s=2000) == EINVAL                    # sink beyond the block
    assert call(m=16, k=65) == EINVAL                # topk * chunk beyond the block
    assert call(mode=7) == EINVAL
    assert call(batch=-1) == EINVAL
    assert call(L=1 << 31, N=1, i=0, s=0, k=0) == EINVAL
    assert call(pos=None) == EINVAL
    assert call(sel=None) == EINVAL                  # Max-IDF prefix of an i > 0 block
    assert call(batch=0, sel=None, pos=None) == 0    # nothing to write
    # no selections needed (these would launch, so only their refusals are
    # checked here): anchor and Even-Spaced modes, block 0, k = 0
    assert call(sel=None, pos=None, mode=2) == EINVAL
    assert call(sel=None, pos=None, i=0) == EINVAL


def test_phase1_gather_validation():
    f = _lib.lib().pulsar_phase1_gather
    def call(X=FAKE, batch=1, L=4096, H=2, d=64, N=4, i=2, s=64, m=16, k=4, sel=FAKE, mode=0,
             pm=1, base=10000.0, out=FAKE):
        return f(X, batch, L, H, d, N, i, s, m, k, sel, mode, pm, None, base, out, None)
    assert call(pm=3) == EINVAL and call(pm=-1) == EINVAL
    assert call(L=4097) == EINVAL
    assert call(i=4) == EINVAL
    assert call(H=0) == EINVAL
    assert call(X=None) == EINVAL and call(out=None) == EINVAL
    assert call(out=FAKE + 2) == EINVAL
    assert call(sel=None) == EINVAL                  # summary mode needs a selection
    assert call(base=0.0) == EINVAL                  # rotating needs a base or table
    assert call(d=96) == EUNSUP and call(d=63) == EINVAL
    assert call(batch=0, X=None, out=None) == 0      # nothing to do


def test_maxidf_workspace_sizes():
    ws = _lib.lib().pulsar_maxidf_workspace_bytes
    # 16 bitmaps of 4008 words and a 128256-byte df table per 128K sequence
    one = ws(1, 131072, 16, 32, 128256)
    assert one == ((16 * 4008 * 4 + 31) // 32) * 32 + 4008 * 32
    assert ws(8, 131072, 16, 32, 128256) == 8 * one
    assert ws(16, 131072, 16, 32, 128256) == 16 * one
    assert ws(17, 131072, 16, 32, 128256) == 0     # one workgroup per sequence is as fast
    assert ws(1, 131072, 1, 32, 128256) == 0       # one block: nothing to split
    assert ws(1, 131072, 16, 32, 200000) > 0       # presence in vocabulary slices
    assert ws(1, 131072, 16, 32, 2000000) == 0     # above the 1310720-id bound
    assert ws(1, 4097, 4, 16, 100) == 0            # invalid shapes take no workspace


def test_chunk_workspace_sizes():
    ws = _lib.lib().pulsar_chunk_workspace_bytes
    mx = _lib.lib().pulsar_maxidf_workspace_bytes
    # the Max-IDF split path's layout, for every scorer
    for scorer in range(4):
        assert ws(1, 131072, 16, 32, 128256, scorer) == mx(1, 131072, 16, 32, 128256)
        assert ws(16, 131072, 16, 32, 128256, scorer) == mx(16, 131072, 16, 32, 128256)
        assert ws(17, 131072, 16, 32, 128256, scorer) == 0
    assert ws(1, 131072, 1, 32, 128256, 1) == 0       # one block: nothing to split
    assert ws(1, 131072, 17, 32, 128256, 1) == 0      # the scorers take at most 16 blocks
    assert ws(1, 131072, 16, 32, 128256, 4) == 0      # unknown scorer
    assert ws(1, 131072, 16, 24, 128256, 1) == 0      # chunk not a power of two
    # no size where the call itself is unsupported (BM25's one-workgroup
    # layout beyond LDS), while TF-IDF, which stages nothing, still fits
    assert ws(1, 131072, 16, 32, 140000, 2) == 0
    assert ws(1, 131072, 16, 32, 140000, 1) > 0


def test_chunk_summaries_validation():
    f = _lib.lib().pulsar_chunk_summaries
    def call(ids=FAKE, batch=1, L=4096, N=4, m=16, k=4, V=1000, scorer=1, sel=FAKE):
        return f(ids, batch, L, N, m, k, V, scorer, sel, None, None, 0, None)
    assert call(scorer=4) == EINVAL and call(scorer=-1) == EINVAL
    assert call(L=4097) == EINVAL          # L % N
    assert call(m=24) == EINVAL            # Lb % m
    assert call(k=65) == EINVAL            # k > Lb / m
    assert call(ids=None) == EINVAL
    assert call(ids=FAKE + 4) == EINVAL    # misaligned
    assert call(sel=None) == EINVAL
    assert call(N=32, L=4096) == EUNSUP    # more than 16 blocks
    assert call(m=512, L=8192, k=1) == EUNSUP
    assert call(L=131072, N=16, m=32, k=4, V=150000, scorer=2) == EUNSUP  # LDS
    assert call(batch=0, ids=None, sel=None) == 0
    # a workspace below the size query
    need = _lib.lib().pulsar_chunk_workspace_bytes(1, 4096, 4, 16, 1000, 1)
    assert need > 0
    assert f(FAKE, 1, 4096, 4, 16, 4, 1000, 1, FAKE, None, FAKE, need - 1, None) == EWS
    assert f(FAKE, 1, 4096, 4, 16, 4, 1000, 1, FAKE, None, FAKE + 8, need, None) == EWS
