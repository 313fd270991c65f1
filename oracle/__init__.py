"""fp64 CPU oracle for Pulsar Attention's Phase-1 / Phase-2 hot path.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plainly written reference
that the HIP library is checked against.  Only the test suite, the smoke check
in ``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import
or call it; the product path (``paper_2607_20457_amd``) never does, and the
oracle imports nothing from the product path.  The two share no code: both
receive their inputs from ``paper_2607_20457_amd.workload``, which only draws
random numbers.

Modules, each following the paper's definitions in its own notation:

* ``maxidf``    -- document frequency, IDF (Eq. idf), Max-IDF chunk score
                   (Eq. 2 / Eq. maxidf), top-k selection in positional order
                   (Algorithm 1, summary step; Appendix "Scoring Heuristic
                   Details").
* ``assembly``  -- causal assembly of the Phase-1 input and its sparse global
                   position ids (Eq. 3; Appendix "RoPE Position ID
                   Assignment"), the Star Attention anchor input, and the
                   retained KV rows (Appendix "KV Cache Discard").
* ``attention`` -- softmax attention (Eq. 1) over the assembled input with an
                   index-causal mask, Phase-2 per-shard partials with
                   log-sum-exp, the online-softmax merge (Appendix "Phase 2
                   Distributed Softmax Merge", Eqs. lse-merge / out-merge) and
                   dense attention over all keys.
* ``cost``      -- the Phase-1 cost model (Table 4; Appendix "Block-to-Host
                   Scalability Analysis").
* ``rope``      -- rotary position embedding of query/key rows at their
                   preserved global positions (Appendix "RoPE Position ID
                   Assignment", sparse mode).
* ``scorers``   -- the other chunk scorers (TF-IDF, BM25, Entropy) with
                   exact scores rounded once to fp32, and the Even-Spaced
                   token offsets (Appendix "Scoring Heuristic Details").

Readings of points the paper leaves open are listed in each function's
docstring.
"""
from . import assembly, attention, cost, maxidf, rope, scorers  # noqa: F401
