"""Python binding of the C ABI: argument marshalling only.

Every function takes and returns torch tensors on a HIP device; torch is
used to allocate the output buffers and to name the current stream.  All
computation happens in the HIP kernels behind ``libpulsar.so``.
"""
from __future__ import annotations

import ctypes
import math

import torch

from . import _lib

PREFIX_SUMMARY = 0
PREFIX_ANCHOR = 1
PREFIX_EVEN = 2
OUT_F32 = 0
OUT_BF16 = 1
POS_SPARSE = 0
POS_CONTIGUOUS = 1
POS_NONE = 2
SCORE_MAXIDF = 0
SCORE_TFIDF = 1
SCORE_BM25 = 2
SCORE_ENTROPY = 3


def _stream():
    return int(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, dtype, name: str):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def maxidf_workspace_bytes(batch: int, L: int, num_blocks: int, chunk: int, vocab: int) -> int:
    return int(_lib.lib().pulsar_maxidf_workspace_bytes(batch, L, num_blocks, chunk, vocab))


def maxidf_summaries(ids: torch.Tensor, num_blocks: int, chunk: int, topk: int, vocab: int,
                     return_mindf: bool = False, return_idf: bool = False, workspace="auto"):
    """Top-k Max-IDF chunks per block.  ids int32 [batch, L] ->
    sel int32 [batch, num_blocks, topk] (+ mindf [batch, N, C], idf [batch, V]).
    workspace: "auto" allocates the split path's workspace when the shapes
    use one, None runs one workgroup per sequence, or a device buffer."""
    if ids.dim() == 1:
        ids = ids[None]
    _need(ids, torch.int32, "ids")
    batch, L = ids.shape
    C = (L // num_blocks) // chunk if num_blocks > 0 and chunk > 0 else 0
    dev = ids.device
    sel = torch.empty((batch, num_blocks, topk), dtype=torch.int32, device=dev)
    mindf = torch.empty((batch, num_blocks, C), dtype=torch.int32, device=dev) if return_mindf else None
    idf = torch.empty((batch, vocab), dtype=torch.float32, device=dev) if return_idf else None
    need = maxidf_workspace_bytes(batch, L, num_blocks, chunk, vocab) if num_blocks > 0 else 0
    if isinstance(workspace, str):
        workspace = torch.empty(need, dtype=torch.uint8, device=dev) if need else None
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.lib().pulsar_maxidf_summaries(_ptr(ids), batch, L, num_blocks, chunk, topk, vocab,
                                            _ptr(sel), _ptr(mindf), _ptr(idf), _ptr(workspace),
                                            ws_bytes, _stream())
    _lib.check(st, "pulsar_maxidf_summaries")
    out = [sel]
    if return_mindf:
        out.append(mindf)
    if return_idf:
        out.append(idf)
    return out[0] if len(out) == 1 else tuple(out)


def chunk_workspace_bytes(batch: int, L: int, num_blocks: int, chunk: int, vocab: int,
                          scorer: int) -> int:
    return int(_lib.lib().pulsar_chunk_workspace_bytes(batch, L, num_blocks, chunk, vocab, scorer))


def chunk_summaries(ids: torch.Tensor, num_blocks: int, chunk: int, topk: int, vocab: int,
                    scorer: int, return_scores: bool = False, workspace="auto"):
    """Top-k chunks per block under a scorer (SCORE_*).  ids int32 [batch, L]
    -> sel int32 [batch, num_blocks, topk] (+ fp32 scores [batch, N, C]).
    workspace: "auto" allocates the split path's workspace when the shapes
    use one, None runs one workgroup per sequence, or a device buffer."""
    if ids.dim() == 1:
        ids = ids[None]
    _need(ids, torch.int32, "ids")
    batch, L = ids.shape
    C = (L // num_blocks) // chunk if num_blocks > 0 and chunk > 0 else 0
    dev = ids.device
    sel = torch.empty((batch, num_blocks, topk), dtype=torch.int32, device=dev)
    scores = torch.empty((batch, num_blocks, C), dtype=torch.float32, device=dev) \
        if return_scores else None
    need = chunk_workspace_bytes(batch, L, num_blocks, chunk, vocab, scorer) \
        if num_blocks > 0 else 0
    if isinstance(workspace, str):
        workspace = torch.empty(need, dtype=torch.uint8, device=dev) if need else None
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.lib().pulsar_chunk_summaries(_ptr(ids), batch, L, num_blocks, chunk, topk, vocab,
                                           scorer, _ptr(sel), _ptr(scores), _ptr(workspace),
                                           ws_bytes, _stream())
    _lib.check(st, "pulsar_chunk_summaries")
    return (sel, scores) if return_scores else sel


def phase1_len(L: int, num_blocks: int, block_idx: int, sink: int, chunk: int, topk: int,
               prefix_mode: int = PREFIX_SUMMARY) -> int:
    n = _lib.lib().pulsar_phase1_len(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode)
    if n < 0:
        _lib.check(int(n), "pulsar_phase1_len")
    return int(n)


def phase1_positions(sel, batch: int, L: int, num_blocks: int, block_idx: int, sink: int,
                     chunk: int, topk: int, prefix_mode: int = PREFIX_SUMMARY,
                     device=None) -> torch.Tensor:
    """Row -> global position map of Input_i, int32 [batch, n_i]."""
    n = phase1_len(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode)
    if sel is not None:
        _need(sel, torch.int32, "sel")
        device = sel.device
    pos = torch.empty((batch, n), dtype=torch.int32, device=device or "cuda")
    st = _lib.lib().pulsar_phase1_positions(_ptr(sel), batch, L, num_blocks, block_idx, sink,
                                            chunk, topk, prefix_mode, _ptr(pos), _stream())
    _lib.check(st, "pulsar_phase1_positions")
    return pos


def _freq_table(inv_freq, d):
    if inv_freq is None:
        return None
    vals = [float(v) for v in (inv_freq.tolist() if hasattr(inv_freq, "tolist") else inv_freq)]
    if len(vals) != d // 2:
        raise ValueError("inv_freq must hold d/2 values")
    return (ctypes.c_float * len(vals))(*vals)


def phase1_gather(X, num_blocks: int, block_idx: int, sink: int, chunk: int, topk: int,
                  sel=None, prefix_mode: int = PREFIX_SUMMARY, pos_mode: int = POS_SPARSE,
                  inv_freq=None, base: float = 500000.0):
    """Block i's assembled input from X bf16 [b, L, H, d], each row rotated
    by its global position (POS_SPARSE), its row index (POS_CONTIGUOUS) or not
    at all (POS_NONE) -> bf16 [b, n_i, H, d]."""
    _need(X, torch.bfloat16, "X")
    if sel is not None:
        _need(sel, torch.int32, "sel")
    b, L, H, d = X.shape
    n = phase1_len(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode)
    out = torch.empty((b, n, H, d), dtype=torch.bfloat16, device=X.device)
    table = _freq_table(inv_freq, d)
    st = _lib.lib().pulsar_phase1_gather(_ptr(X), b, L, H, d, num_blocks, block_idx, sink, chunk,
                                         topk, _ptr(sel), prefix_mode, pos_mode,
                                         None if table is None else
                                         ctypes.cast(table, ctypes.c_void_p),
                                         float(base), _ptr(out), _stream())
    _lib.check(st, "pulsar_phase1_gather")
    return out


def phase1_attn(Q, K, V, num_blocks: int, block_idx: int, sink: int, chunk: int, topk: int,
                sel=None, prefix_mode: int = PREFIX_SUMMARY, softmax_scale: float | None = None,
                o_dtype: int = OUT_F32, return_lse: bool = True, keep_kv: bool = False,
                out=None):
    """Phase-1 causal attention over Input_i.  Q bf16 [b, L, Hq, d], K/V bf16
    [b, L, Hkv, d] -> O [b, n_i, Hq, d] (+ lse [b, Hq, n_i], K_keep, V_keep)."""
    for t, name in ((Q, "Q"), (K, "K"), (V, "V")):
        _need(t, torch.bfloat16, name)
    if sel is not None:
        _need(sel, torch.int32, "sel")
    b, L, Hq, d = Q.shape
    Hkv = K.shape[2]
    if K.shape != (b, L, Hkv, d) or V.shape != K.shape:
        raise ValueError("K and V must be [batch, L, Hkv, d] matching Q")
    n = phase1_len(L, num_blocks, block_idx, sink, chunk, topk, prefix_mode)
    scale = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    dev = Q.device
    if out is not None:
        O = out
        _need(O, torch.bfloat16 if o_dtype == OUT_BF16 else torch.float32, "out")
        if O.shape != (b, n, Hq, d):
            raise ValueError("out has the wrong shape")
    else:
        O = torch.empty((b, n, Hq, d), device=dev,
                        dtype=torch.bfloat16 if o_dtype == OUT_BF16 else torch.float32)
    lse = torch.empty((b, Hq, n), dtype=torch.float32, device=dev) if return_lse else None
    Lb = L // num_blocks
    Kk = torch.empty((b, Lb, Hkv, d), dtype=torch.bfloat16, device=dev) if keep_kv else None
    Vk = torch.empty((b, Lb, Hkv, d), dtype=torch.bfloat16, device=dev) if keep_kv else None
    st = _lib.lib().pulsar_phase1_attn(_ptr(Q), _ptr(K), _ptr(V), b, L, Hq, Hkv, d, num_blocks,
                                       block_idx, sink, chunk, topk, _ptr(sel), prefix_mode,
                                       scale, _ptr(O), o_dtype, _ptr(lse), _ptr(Kk), _ptr(Vk),
                                       _stream())
    _lib.check(st, "pulsar_phase1_attn")
    res = [O]
    if return_lse:
        res.append(lse)
    if keep_kv:
        res += [Kk, Vk]
    return res[0] if len(res) == 1 else tuple(res)


def phase2_workspace_bytes(n_shards: int, Tq: int, S: int, Hq: int, Hkv: int, d: int) -> int:
    return int(_lib.lib().pulsar_phase2_workspace_bytes(n_shards, Tq, S, Hq, Hkv, d))


def phase2_partial(q, K, V, softmax_scale: float | None = None, workspace=None):
    """Per-shard partials.  q bf16 [Tq, Hq, d]; K/V bf16 [n_shards, S, Hkv, d]
    -> (o_parts f32 [n_shards, Tq, Hq, d], lse_parts f32 [n_shards, Hq, Tq])."""
    _need(q, torch.bfloat16, "q")
    _need(K, torch.bfloat16, "K")
    _need(V, torch.bfloat16, "V")
    Tq, Hq, d = q.shape
    H, S, Hkv, dk = K.shape
    if dk != d or V.shape != K.shape:
        raise ValueError("K/V must be [n_shards, S, Hkv, d]")
    scale = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    dev = q.device
    o = torch.empty((H, Tq, Hq, d), dtype=torch.float32, device=dev)
    lse = torch.empty((H, Hq, Tq), dtype=torch.float32, device=dev)
    need = phase2_workspace_bytes(H, Tq, S, Hq, Hkv, d)
    if need and (workspace is None or workspace.numel() * workspace.element_size() < need):
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    st = _lib.lib().pulsar_phase2_partial(_ptr(q), _ptr(K), _ptr(V), H, Tq, S, Hq, Hkv, d, scale,
                                          _ptr(o), _ptr(lse), _ptr(workspace),
                                          need, _stream())
    _lib.check(st, "pulsar_phase2_partial")
    return o, lse


def lse_merge(o_parts, lse_parts):
    """Merge H partials: o_parts f32 [H, Tq, Hq, d], lse_parts f32 [H, Hq, Tq]
    -> (o [Tq, Hq, d], lse [Hq, Tq])."""
    _need(o_parts, torch.float32, "o_parts")
    _need(lse_parts, torch.float32, "lse_parts")
    H, Tq, Hq, d = o_parts.shape
    if lse_parts.shape != (H, Hq, Tq):
        raise ValueError("lse_parts must be [H, Hq, Tq]")
    o = torch.empty((Tq, Hq, d), dtype=torch.float32, device=o_parts.device)
    lse = torch.empty((Hq, Tq), dtype=torch.float32, device=o_parts.device)
    st = _lib.lib().pulsar_lse_merge(_ptr(o_parts), _ptr(lse_parts), H, Tq, Hq, d, _ptr(o),
                                     _ptr(lse), _stream())
    _lib.check(st, "pulsar_lse_merge")
    return o, lse


def rope_(x, pos=None, pos_offset: int = 0, inv_freq=None, base: float = 500000.0):
    """Rotate x bf16 [batch, n, H, d] (or [n, H, d]) in place by the rows'
    positions: pos int32 [batch, n] (None: row index) plus pos_offset.
    inv_freq: the d/2 frequencies (a host sequence of floats), or None for
    base^(-2i/d).  Returns x."""
    _need(x, torch.bfloat16, "x")
    xv = x[None] if x.dim() == 3 else x
    batch, n, H, d = xv.shape
    if pos is not None:
        _need(pos, torch.int32, "pos")
        if pos.numel() != batch * n:
            raise ValueError("pos must hold one position per row")
    table = _freq_table(inv_freq, d)
    st = _lib.lib().pulsar_rope(_ptr(xv), batch, n, H, d, _ptr(pos), int(pos_offset),
                                None if table is None else ctypes.cast(table, ctypes.c_void_p),
                                float(base), _stream())
    _lib.check(st, "pulsar_rope")
    return x


def phase2_query(q, Kg, Vg, G: int, K=None, V=None, softmax_scale: float | None = None,
                 workspace=None):
    """Attention of Tq new tokens: q bf16 [Tq, Hq, d] over the retained
    shards K/V bf16 [n_shards, S, Hkv, d] (or None) and the generation shard's
    appended rows Kg/Vg bf16 [G + Tq, Hkv, d] up to each token itself
    -> (o f32 [Tq, Hq, d], lse f32 [Hq, Tq])."""
    _need(q, torch.bfloat16, "q")
    _need(Kg, torch.bfloat16, "Kg")
    _need(Vg, torch.bfloat16, "Vg")
    Tq, Hq, d = q.shape
    Hkv = Kg.shape[1]
    if Kg.shape != (G + Tq, Hkv, d) or Vg.shape != Kg.shape:
        raise ValueError("Kg/Vg must be [G + Tq, Hkv, d]")
    n_shards, S = 0, 0
    if K is not None:
        _need(K, torch.bfloat16, "K")
        _need(V, torch.bfloat16, "V")
        n_shards, S = K.shape[0], K.shape[1]
        if K.shape != (n_shards, S, Hkv, d) or V.shape != K.shape:
            raise ValueError("K/V must be [n_shards, S, Hkv, d]")
    scale = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    dev = q.device
    o = torch.empty((Tq, Hq, d), dtype=torch.float32, device=dev)
    lse = torch.empty((Hq, Tq), dtype=torch.float32, device=dev)
    need = _lib.lib().pulsar_phase2_query_workspace_bytes(n_shards, Tq, S, G, Hq, Hkv, d)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    st = _lib.lib().pulsar_phase2_query(_ptr(q), _ptr(Kg), _ptr(Vg), G, _ptr(K), _ptr(V), n_shards,
                                        Tq, S, Hq, Hkv, d, scale, _ptr(o), _ptr(lse),
                                        _ptr(workspace), need, _stream())
    _lib.check(st, "pulsar_phase2_query")
    return o, lse


def phase2_query_noalloc(q, Kg, Vg, G: int, K=None, V=None, softmax_scale: float | None = None):
    """``phase2_query`` through the entry point that allocates nothing: the
    partials live in the library's static per-device scratch.  The outputs
    are allocated here by torch, as for every binding."""
    _need(q, torch.bfloat16, "q")
    _need(Kg, torch.bfloat16, "Kg")
    _need(Vg, torch.bfloat16, "Vg")
    Tq, Hq, d = q.shape
    Hkv = Kg.shape[1]
    if Kg.shape != (G + Tq, Hkv, d) or Vg.shape != Kg.shape:
        raise ValueError("Kg/Vg must be [G + Tq, Hkv, d]")
    n_shards, S = 0, 0
    if K is not None:
        _need(K, torch.bfloat16, "K")
        _need(V, torch.bfloat16, "V")
        n_shards, S = K.shape[0], K.shape[1]
        if K.shape != (n_shards, S, Hkv, d) or V.shape != K.shape:
            raise ValueError("K/V must be [n_shards, S, Hkv, d]")
    scale = 1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale
    o = torch.empty((Tq, Hq, d), dtype=torch.float32, device=q.device)
    lse = torch.empty((Hq, Tq), dtype=torch.float32, device=q.device)
    st = _lib.lib().pulsar_phase2_query_noalloc(_ptr(q), _ptr(Kg), _ptr(Vg), G, _ptr(K), _ptr(V),
                                                n_shards, Tq, S, Hq, Hkv, d, scale, _ptr(o),
                                                _ptr(lse), _stream())
    _lib.check(st, "pulsar_phase2_query_noalloc")
    return o, lse
