"""Pulsar Attention Phase-1 / Phase-2 hot path for MI355X (gfx950).

The computation lives in ``libpulsar.so`` (HIP kernels behind the C ABI of
``include/pulsar.h``); ``api`` is its thin torch-facing binding and
``workload`` draws the seeded synthetic inputs.
"""
from .api import (OUT_BF16, OUT_F32, POS_CONTIGUOUS, POS_NONE, POS_SPARSE,  # noqa: F401
                  PREFIX_ANCHOR, PREFIX_EVEN, PREFIX_SUMMARY, SCORE_BM25,
                  SCORE_ENTROPY, SCORE_MAXIDF, SCORE_TFIDF, chunk_summaries,
                  chunk_workspace_bytes, lse_merge, maxidf_summaries, maxidf_workspace_bytes,
                  phase1_attn, phase1_gather, phase1_len, phase1_positions, phase2_partial,
                  phase2_query, phase2_query_noalloc, phase2_workspace_bytes, rope_)
