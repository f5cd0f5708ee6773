"""Stage (a) oracle: chunk prefill, chunk cache, key summary, eviction score.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows Section 5.1 ("Chunk Prefill", Eq. 2) and Section 5.2 ("Intra-chunk
sparsity", Eq. 5) of the paper.  Readings taken where the paper is silent:

* A BOS token is prepended to every chunk (Section 5.1) and its KV row is kept
  in the chunk cache at slot 0, so the cache holds 1+C rows per chunk.
* The chunk sequence is [BOS; c_1..c_C; q_1..q_Lq; m_1..m_Lm] and attention
  inside it is fully bidirectional with no mask; nothing attends across chunks.
* Attn(x, y) in Eq. 5 is the softmax probability of row x on column y in the
  chunk-local forward, normalised over all S_c = 1+C+Lq+Lm columns, with the
  default scale 1/sqrt(d).  Eq. 5 has no head index: the score is summed over
  all query heads, so one token set per (sequence, chunk) serves every head.
* Only the L_q query rows enter Eq. 5; the L_m pseudo-label rows only take
  part in the normalisation.  BOS is not a candidate token.
* The chunk key summary used by the per-step chunk score is the mean of the C
  content keys of the chunk (BOS excluded), per KV head.
* The query-to-chunk variant of the token score (the paper's ablation of the
  retention score) keeps only the first sum of Eq. 5: the mass the query rows
  put on the token.
* The content mass of a query or pseudo-label row is the probability it puts
  on the C content columns of its chunk (BOS excluded); the prefill-time chunk
  score (``oracle.chunk_score``) is built from it.

Layouts (numpy, any float dtype on input, float64 inside):
  q_pre (B, N, 1+C, Hq, d), k_pre / v_pre (B, N, 1+C, Hkv, d), slot 0 = BOS;
  q_qm (B, Lq+Lm, Hq, d) shared by all chunks, or (B, N, Lq+Lm, Hq, d);
  k_qm / v_qm likewise with Hkv heads.
"""

import numpy as np


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def chunk_rows(x_pre, x_qm, b, n, head):
    """Rows of chunk n's sequence [BOS; c; q; m] for one head, float64 (S_c, d).

    The q/m rows come from the shared (B, Lq+Lm, H, d) tensor, or from chunk n's
    slice when the tensor carries a chunk axis.
    """
    pre = _f64(x_pre[b, n, :, head, :])
    qm = x_qm[b, n] if x_qm.ndim == 5 else x_qm[b]
    return np.concatenate([pre, _f64(qm[:, head, :])], axis=0)


def chunk_probs(q_rows, k_rows, scale):
    """Softmax probabilities of one chunk forward, two-pass, float64.

    S = scale * Q K^T over every row pair of the chunk sequence (no mask);
    P = exp(S - rowmax) / rowsum.  Also returns the natural-log row LSE.
    """
    s = scale * (q_rows @ k_rows.T)
    m = s.max(axis=1, keepdims=True)
    ex = np.exp(s - m)
    z = ex.sum(axis=1, keepdims=True)
    p = ex / z
    lse = (m + np.log(z))[:, 0]
    return p, lse


def prefill_unit_ref(q_pre, k_pre, v_pre, q_qm, k_qm, v_qm, b, n, h, q_len, scale=None):
    """One (sequence b, chunk n, query head h) of the chunk prefill.

    Returns a dict with
      o      (S_c, d)  attention output rows, ordered BOS, c, q, m (Eq. 2 forward);
      p      (S_c, S_c) the probabilities;
      lse    (S_c,)    natural-log row LSE;
      e_head (C,)      this head's contribution to Eq. 5 for the C content tokens;
      e_q2c_head (C,)  its first sum only (query rows -> content columns);
      content_mass (Lq+Lm,) mass of each q/m row on the C content columns.
    """
    hq, hkv = q_pre.shape[3], k_pre.shape[3]
    d = q_pre.shape[4]
    c1 = q_pre.shape[2]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(d)
    g = h // (hq // hkv)
    qr = chunk_rows(q_pre, q_qm, b, n, h)
    kr = chunk_rows(k_pre, k_qm, b, n, g)
    vr = chunk_rows(v_pre, v_qm, b, n, g)
    p, lse = chunk_probs(qr, kr, scale)
    o = p @ vr
    content = slice(1, c1)            # slots 1..C
    qrows = slice(c1, c1 + q_len)     # the L_q query rows
    # Eq. 5: query row -> content column, plus content row -> query column.
    e_q2c_head = p[qrows, content].sum(axis=0)
    e_head = e_q2c_head + p[content, qrows].sum(axis=1)
    content_mass = p[c1:, content].sum(axis=1)
    return {"o": o, "p": p, "lse": lse, "e_head": e_head, "e_q2c_head": e_q2c_head,
            "content_mass": content_mass}


def cache_ref(x_pre):
    """Chunk cache of one layer: (B, N, 1+C, H, d) -> (B, N, H, 1+C, d).

    An exact copy in the input dtype (no rounding): every chunk's BOS and
    content KV rows are stored once, chunk-contiguous per head.
    """
    return np.ascontiguousarray(np.transpose(np.asarray(x_pre), (0, 1, 3, 2, 4)))


def key_mean_ref(k_pre):
    """Chunk key summary: mean of the C content keys (slots 1..C), (B, N, Hkv, d)."""
    return _f64(k_pre)[:, :, 1:, :, :].mean(axis=2)


def prefill_ref(q_pre, k_pre, v_pre, q_qm, k_qm, v_qm, q_len, scale=None):
    """Whole stage (a) for small inputs.

    Returns dict: o (B, N, S_c, Hq, d), k_cache / v_cache (B, N, Hkv, 1+C, d,
    input dtype), tok_score (B, N, C) = Eq. 5 summed over heads,
    tok_score_q2c (B, N, C) = its first sum only, key_mean (B, N, Hkv, d),
    lse (B, N, Hq, S_c), content_mass (B, N, Hq, Lq+Lm).
    """
    bsz, nch, c1, hq, d = q_pre.shape
    lqm = q_qm.shape[-3]
    sc = c1 + lqm
    o = np.zeros((bsz, nch, sc, hq, d))
    lse = np.zeros((bsz, nch, hq, sc))
    tok = np.zeros((bsz, nch, c1 - 1))
    tok_q2c = np.zeros((bsz, nch, c1 - 1))
    mass = np.zeros((bsz, nch, hq, lqm))
    for b in range(bsz):
        for n in range(nch):
            for h in range(hq):
                u = prefill_unit_ref(q_pre, k_pre, v_pre, q_qm, k_qm, v_qm, b, n, h, q_len, scale)
                o[b, n, :, h, :] = u["o"]
                lse[b, n, h] = u["lse"]
                tok[b, n] += u["e_head"]
                tok_q2c[b, n] += u["e_q2c_head"]
                mass[b, n, h] = u["content_mass"]
    return {
        "o": o,
        "k_cache": cache_ref(k_pre),
        "v_cache": cache_ref(v_pre),
        "tok_score": tok,
        "tok_score_q2c": tok_q2c,
        "key_mean": key_mean_ref(k_pre),
        "lse": lse,
        "content_mass": mass,
    }
