"""Stage (b) oracle: per-step chunk score, top-K chunks, top-B tokens.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 5.2 keeps the K best chunks ("inter-chunk sparsity") and, inside each
kept chunk, the B tokens with the highest eviction score of Eq. 5
("intra-chunk sparsity").  The paper ranks chunks by a language-model NLL
(Eqs. 3-4), which an attention-only slice cannot evaluate.  The reading taken
here is an attention-space proxy computed at every denoising step:

    qbar_h = (1/L_d) * sum_r Q_dec[r, h]                  (mean decode query)
    s_n    = sum_h scale * <qbar_h, kbar[n, g(h)]>         (higher = kept)

with kbar the chunk key summary of stage (a) and g(h) = h // (Hq/Hkv).
Ties rank the lower index first for chunks and tokens alike, and both lists
are returned in ascending order.  Token lists hold cache slots 1..C (slot 0 is
the chunk's BOS row, which every kept chunk contributes on top of the B
tokens).

The chunk score is pinned to the definition above (worked example, zero
query, linearity, GQA group mapping); against the paper it is parity
unpinned: the paper prints no value of this proxy.
"""

import numpy as np


def chunk_scores_ref(q_dec, key_mean, scale=None):
    """Chunk scores s (B, N) from decode queries (B, Ld, Hq, d) and key means (B, N, Hkv, d)."""
    q = np.asarray(q_dec, dtype=np.float64)
    kbar = np.asarray(key_mean, dtype=np.float64)
    bsz, _, hq, d = q.shape
    nch, hkv = kbar.shape[1], kbar.shape[2]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(d)
    qbar = q.mean(axis=1)                     # (B, Hq, d)
    s = np.zeros((bsz, nch))
    for b in range(bsz):
        for n in range(nch):
            for h in range(hq):
                g = h // (hq // hkv)
                s[b, n] += scale * float(qbar[b, h] @ kbar[b, n, g])
    return s


def topk_ref(x, k):
    """Indices of the k largest entries of x, ties to the lower index, ascending."""
    x = np.asarray(x, dtype=np.float64)
    order = np.lexsort((np.arange(x.shape[0]), -x))   # primary: -x, secondary: index
    return np.sort(order[:k])


def token_rank_ref(tok_score):
    """Rank of every token inside its chunk by Eq. 5 score: 0 = highest, ties to
    the lower index (Section 5.2: tokens are ranked by eviction score).
    tok_score (B, N, C) -> int32 (B, N, C)."""
    e = np.asarray(tok_score, dtype=np.float64)
    bsz, nch, c = e.shape
    rank = np.zeros((bsz, nch, c), dtype=np.int32)
    for b in range(bsz):
        for n in range(nch):
            order = np.lexsort((np.arange(c), -e[b, n]))
            rank[b, n, order] = np.arange(c, dtype=np.int32)
    return rank


def tokens_by_rank_ref(tok_rank, chunk_idx, tok_budget):
    """Kept slots of each selected chunk: the tokens ranked below tok_budget, as
    ascending cache slots 1 + j.  Returns int32 (B, K, Btok)."""
    r = np.asarray(tok_rank)
    ci = np.asarray(chunk_idx)
    out = np.zeros(ci.shape + (tok_budget,), dtype=np.int32)
    for b in range(ci.shape[0]):
        for kk, n in enumerate(ci[b]):
            out[b, kk] = 1 + np.nonzero(r[b, n] < tok_budget)[0]
    return out


def score_select_ref(q_dec, key_mean, tok_score, top_k, tok_budget, scale=None):
    """Whole stage (b) for one step.

    Returns chunk_idx (B, K) int32 ascending, tok_slot (B, K, Btok) int32
    ascending cache slots in 1..C, and the chunk scores (B, N).
    """
    s = chunk_scores_ref(q_dec, key_mean, scale)
    e = np.asarray(tok_score, dtype=np.float64)
    bsz = s.shape[0]
    chunk_idx = np.zeros((bsz, top_k), dtype=np.int32)
    tok_slot = np.zeros((bsz, top_k, tok_budget), dtype=np.int32)
    for b in range(bsz):
        chunk_idx[b] = topk_ref(s[b], top_k)
        for kk, n in enumerate(chunk_idx[b]):
            tok_slot[b, kk] = 1 + topk_ref(e[b, n], tok_budget)
    return chunk_idx, tok_slot, s
