"""Plain, slow float64 CPU oracle of the Prefilling-dLLM block-sparse attention path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or run
anything in this package: only the test suite, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the
HIP library (no kernels, headers, helpers or generated tables) and imports
nothing from it.

Every function works on numpy arrays holding the exact values the GPU path
receives (bf16 or fp32 inputs upcast exactly to float64) and computes in
float64 with materialised score matrices and an explicit two-pass softmax, so
that each step can be checked against the paper by eye:

* ``prefill``  -- stage (a): chunk prefill (Section 5.1, Eq. 2), the chunk
  cache, the chunk key summary and the intra-chunk eviction score (Section 5.2,
  Eq. 5).
* ``select``   -- stage (b): chunk scores, top-K chunks and top-B tokens per
  kept chunk (Section 5.2, inter- and intra-chunk sparsity).
* ``decode``   -- stage (c): attention of the decode block over the selected
  prefix KV, the static query KV and its own KV (Section 5.3, prefix reuse).
* ``static``   -- static-selection mode: selection once from the pseudo-label
  rows, the kept rows compacted into a contiguous buffer, decode over it.
* ``chunk_score`` -- the prefill-time chunk score built from the attention
  mass the query and pseudo-label rows put on the chunk content (an
  attention-space reading of Eqs. 3-4), and selection of the K lowest.
* ``full_mask`` -- full-mask cache construction: the kept rows and the query
  rows rotated to continuous positions and encoded jointly.

Parity status of each function is stated in its docstring ("pinned by ...").
"""

from .prefill import (
    chunk_rows,
    chunk_probs,
    prefill_unit_ref,
    prefill_ref,
    cache_ref,
    key_mean_ref,
)
from .select import chunk_scores_ref, topk_ref, score_select_ref, token_rank_ref, tokens_by_rank_ref
from .decode import decode_kv_rows, decode_unit_ref, decode_ref
from .static import (
    pseudo_label_queries,
    static_select_ref,
    gather_selected_ref,
    decode_compact_unit_ref,
    decode_compact_ref,
)
from .chunk_score import prefill_chunk_score_ref, select_ranked_ref
from .full_mask import rope_rotate_ref, joint_deltas, joint_rows_ref, joint_attention_ref

__all__ = [
    "chunk_rows",
    "chunk_probs",
    "prefill_unit_ref",
    "prefill_ref",
    "cache_ref",
    "key_mean_ref",
    "chunk_scores_ref",
    "topk_ref",
    "score_select_ref",
    "token_rank_ref",
    "tokens_by_rank_ref",
    "decode_kv_rows",
    "decode_unit_ref",
    "decode_ref",
    "pseudo_label_queries",
    "static_select_ref",
    "gather_selected_ref",
    "decode_compact_unit_ref",
    "decode_compact_ref",
    "prefill_chunk_score_ref",
    "select_ranked_ref",
    "rope_rotate_ref",
    "joint_deltas",
    "joint_rows_ref",
    "joint_attention_ref",
]
