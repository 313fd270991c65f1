"""Seeded synthetic inputs shared by the HIP path and the fp64 oracle.

This module draws random numbers and nothing else: it holds none of the
method's arithmetic (no document frequencies, scores, selection, assembly or
attention).  Both sides receive the arrays it returns, so they see the same
token ids and the same bf16-rounded Q/K/V values.

Workload recipe (stand-ins for the paper's long-context benchmarks, whose
items are not used):

* token ids: truncated Zipf(s) over ranks 1..V with P(r) proportional to r^-s,
  id = r - 1, drawn by inverse-CDF sampling from a PCG64 generator.  The
  unbounded ``numpy.random.zipf`` is not used: rejecting its tail would change
  the law.
* needles: ids that do not occur in the sample, written once each at distinct
  uniformly drawn positions, so that each needle has document frequency 1.
* Q/K/V: float32 N(0,1) from PCG64, rounded to bfloat16 with round-to-nearest-
  even, returned as the raw uint16 bit patterns in ``[batch, L, heads, d]``.
  The flat array is drawn in pieces of 2^24 values; piece j comes from its own
  PCG64 stream seeded with (seed, j), so the pieces can be drawn by several
  threads and the result does not depend on how many.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

__all__ = [
    "zipf_ids",
    "plant_needles",
    "bf16_normal",
    "bf16_bits_to_f32",
    "f32_to_bf16_bits",
    "Config",
    "CONFIGS",
    "make_ids",
    "make_qkv",
]


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def zipf_ids(seed: int, n: int, vocab: int, s: float = 1.1) -> np.ndarray:
    """``n`` int32 ids from a Zipf(s) law truncated to ``vocab`` ranks."""
    rng = _rng(seed)
    w = np.arange(1, vocab + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = rng.random(n)
    ids = np.searchsorted(cdf, u, side="right")
    np.minimum(ids, vocab - 1, out=ids)
    return ids.astype(np.int32)


def plant_needles(seed: int, ids: np.ndarray, count: int, vocab: int):
    """Overwrite ``count`` seeded positions of a 1-D id array with distinct ids
    absent from it.  Returns (ids, needle_ids, positions)."""
    rng = _rng(seed)
    ids = ids.copy()
    present = np.zeros(vocab, dtype=bool)
    present[ids] = True
    absent = np.flatnonzero(~present)
    if absent.size < count:
        raise ValueError("not enough unused ids to plant needles")
    needle_ids = rng.choice(absent, size=count, replace=False).astype(np.int32)
    pos = np.sort(rng.choice(ids.size, size=count, replace=False))
    ids[pos] = needle_ids
    return ids, needle_ids, pos


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest-even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


PIECE = 1 << 24  # values per independently seeded piece of a bf16_normal draw


def bf16_normal(seed: int, shape, scale: float = 1.0) -> np.ndarray:
    """bf16 bit patterns of ``scale * N(0,1)`` float32 samples."""
    out = np.empty(int(np.prod(shape, dtype=np.int64)), dtype=np.uint16)

    def piece(j: int) -> None:
        lo = j * PIECE
        hi = min(out.size, lo + PIECE)
        rng = np.random.Generator(np.random.PCG64([seed, j]))
        x = rng.standard_normal(size=hi - lo, dtype=np.float32)
        if scale != 1.0:
            x *= np.float32(scale)
        out[lo:hi] = f32_to_bf16_bits(x)

    n_pieces = (out.size + PIECE - 1) // PIECE
    workers = max(1, min(n_pieces, len(os.sched_getaffinity(0)), 16))
    if workers == 1:
        for j in range(n_pieces):
            piece(j)
    else:
        with _cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(piece, range(n_pieces)))
    return out.reshape(shape)


@dataclasses.dataclass(frozen=True)
class Config:
    """Shapes of one synthetic workload (Llama-3.1-8B-shaped layer unless noted)."""
    name: str
    L: int
    vocab: int
    num_blocks: int
    sink: int
    chunk: int
    topk: int
    Hq: int
    Hkv: int
    d: int
    batch: int = 1
    needles: int = 0
    zipf_s: float = 1.1
    seed: int = 1000

    @property
    def Lb(self) -> int:
        return self.L // self.num_blocks


# The five workloads, as (name, shapes).  Seeds follow 1000 + workload number.
CONFIGS = {
    "tiny": Config("tiny", L=4096, vocab=32000, num_blocks=4, sink=64, chunk=16,
                   topk=4, Hq=4, Hkv=1, d=64, seed=1001),
    "llama8b_32k": Config("llama8b_32k", L=32768, vocab=128256, num_blocks=8, sink=64,
                          chunk=32, topk=16, Hq=32, Hkv=8, d=128, needles=16, seed=1002),
    "llama8b_128k": Config("llama8b_128k", L=131072, vocab=128256, num_blocks=16, sink=64,
                           chunk=32, topk=32, Hq=32, Hkv=8, d=128, seed=1003),
    "phase2_128k": Config("phase2_128k", L=131072, vocab=128256, num_blocks=16, sink=64,
                          chunk=32, topk=32, Hq=32, Hkv=8, d=128, seed=1004),
    "sweep_128k_b4": Config("sweep_128k_b4", L=131072, vocab=128256, num_blocks=16, sink=64,
                            chunk=32, topk=32, Hq=32, Hkv=8, d=128, batch=4, seed=1005),
}


def make_ids(cfg: Config, batch: int | None = None, vocab: int | None = None) -> np.ndarray:
    """int32 ids ``[batch, L]``: one seeded Zipf sequence per batch row,
    with ``cfg.needles`` needles planted per row."""
    batch = cfg.batch if batch is None else batch
    vocab = cfg.vocab if vocab is None else vocab
    rows = []
    for b in range(batch):
        ids = zipf_ids(cfg.seed * 1000 + b, cfg.L, vocab, cfg.zipf_s)
        if cfg.needles:
            ids, _, _ = plant_needles(cfg.seed * 1000 + 500 + b, ids, cfg.needles, vocab)
        rows.append(ids)
    return np.stack(rows).astype(np.int32)


def make_qkv(cfg: Config, batch: int | None = None, L: int | None = None, q_scale: float = 1.0):
    """bf16 bit patterns ``Q [b,L,Hq,d]``, ``K, V [b,L,Hkv,d]``."""
    batch = cfg.batch if batch is None else batch
    L = cfg.L if L is None else L
    q = bf16_normal(cfg.seed * 10 + 1, (batch, L, cfg.Hq, cfg.d), q_scale)
    k = bf16_normal(cfg.seed * 10 + 2, (batch, L, cfg.Hkv, cfg.d))
    v = bf16_normal(cfg.seed * 10 + 3, (batch, L, cfg.Hkv, cfg.d))
    return q, k, v
