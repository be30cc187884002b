"""CPU oracle for expert-map matching and prefetch-set selection.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only the test suite, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP path
(no kernels, headers, helpers or constant tables) and imports nothing from it.

It is a plain, slow, obviously correct restatement of what the paper defines:

* ``finemoe``  NumPy float64 implementation of semantic and trajectory cosine
  search (Eq. 4, Eq. 5), ranking by highest score, the per-layer trajectory
  re-search schedule of one pass (Section 4.2.2), the redundancy score and
  victim choice of store deduplication (Section 4.4), the optional
  similarity-weighted blend, the similarity-aware threshold of Section 4.3,
  the minimum-cardinality prefetch set of Eq. 6-8, the prefetch and
  eviction priorities of Section 4.5 and the miss indicator of Section 3.
* ``brute``    pure-Python brute force with correctly rounded sums
  (``math.fsum``) and full subset enumeration, used to pin ``finemoe`` on
  tiny inputs.

Every function is pinned by the ``-m "not gpu"`` tests against closed forms,
invariants and brute force, including the similarity-weighted blend with
missing matches and NaN weights (against a correctly rounded blend) and the
searches and redundancy scores over several store chunks (with the chunk size
made small, against brute force over the whole store).  Each pin is chosen so
that a planted mistake in the function it covers makes it fail.
"""
from . import finemoe, brute  # noqa: F401
from .finemoe import (  # noqa: F401
    widen, cosine, trajectory_scores, semantic_scores, rank, match_trajectory,
    match_semantic, research_schedule, redundancy, dedup_slots, insert_dedup, threshold, select_row, blend_rows, select_prefetch, guide_row, priority_order, activated, miss_counts,
    TAU_FIXED, TAU_DYNAMIC, BLEND_NONE, BLEND_SCORE, PRI_PREFETCH, PRI_EVICT,
)
