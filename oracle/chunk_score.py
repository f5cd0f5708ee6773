"""Prefill-time chunk score and selection from given chunk scores.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 5.1 scores every chunk during its own prefill forward with two
length-normalised negative log-likelihoods: of the query window given the
chunk (Eq. 3, s_I) and of the pseudo-labels given the chunk and the query
(Eq. 4, s_P).  Section 5.2 ("Inter-chunk sparsity") adds the two with equal
weight and keeps the K chunks with the LOWEST sum.  Both terms need the
language-model head, which an attention-only slice does not have.  The reading
taken here keeps their form -- a length-normalised negative log of how much a
row draws on the chunk -- and takes for the row's probability the attention
mass it puts on the chunk's content in the same forward:

    a_h(r) = sum_{j = 1..C} P_h[r, j]        row r of the q/m block, head h, BOS excluded
    a(r)   = (1 / H_q) sum_h a_h(r)          head-averaged mass (one value per layer)
    s_I    = -(1 / L_q) sum_{r in q} ln a(r)
    s_P    = -(1 / L_m) sum_{r in m} ln a(r)     (0 when L_m = 0)
    s      = s_I + s_P                            lower = kept

a_h comes from ``oracle.prefill`` (``content_mass``).  Ties in the selection
rank the lower chunk index first; the kept lists are ascending.

Pinned by: a hand-derived two-head example, the one-head prefill example, the
closed form for all-zero queries, the dense block-diagonal forward of all
chunks, and subset enumeration for the K lowest.  Against the paper itself
the score is parity unpinned: the paper prints no value of this reading.
"""

import numpy as np

from . import select as _select


def prefill_chunk_score_ref(content_mass, q_len):
    """Chunk scores (B, N) from the per-head content masses (B, N, Hq, Lq+Lm).

    Rows 0..q_len-1 of the last axis are the query rows, the rest the
    pseudo-label rows.
    """
    a = np.asarray(content_mass, dtype=np.float64).mean(axis=2)   # (B, N, Lq+Lm): head average
    with np.errstate(divide="ignore"):
        nll = -np.log(a)
    s_i = nll[..., :q_len].mean(axis=-1)
    s_p = nll[..., q_len:].mean(axis=-1) if a.shape[-1] > q_len else np.zeros(s_i.shape)
    return s_i + s_p


def select_ranked_ref(chunk_score, tok_rank, top_k, tok_budget, lowest=True):
    """Top-K chunks by a given score (the K lowest, or the K highest when
    lowest=False; ties to the lower index) and the kept token slots of each.

    chunk_score (B, N), tok_rank (B, N, C) -> chunk_idx (B, K) int32 ascending,
    tok_slot (B, K, Btok) int32 ascending slots in 1..C.
    """
    s = np.asarray(chunk_score, dtype=np.float64)
    key = -s if lowest else s
    chunk_idx = np.stack([_select.topk_ref(key[b], top_k) for b in range(s.shape[0])]).astype(np.int32)
    return chunk_idx, _select.tokens_by_rank_ref(tok_rank, chunk_idx, tok_budget)
