"""Full-mask cache construction: kept rows re-encoded jointly at continuous positions.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 6 (implementation details and the ablation of the KV cache
construction strategy): after selection, the kept chunks and the query are
encoded jointly with the same bidirectional mask as in decoding, the kept
chunks at continuous positions and the query placed after them.  In a
one-layer attention slice that amounts to (readings taken here):

* positions -- the chunk forward gave cache slot s of every chunk position s
  (BOS at 0, content 1..C) and query row j position C+1+j.  In the joint
  layout the k-th kept chunk (ascending chunk order) starts at k*(C+1), so
  each of its rows moves by delta = k*(C+1); the query rows follow the K kept
  chunks, so they move by delta = (K-1)*(C+1).  Rows dropped by intra-chunk
  sparsity leave gaps: kept tokens keep their slot offsets.
* rotary embedding -- rotate-half pairing: dimension i < d/2 pairs with
  i + d/2 at frequency theta_i = base^(-2i/d); moving a row by delta rotates
  every pair by delta*theta_i.  Queries and keys move, values do not.  base = 0
  means no rotation (positions already continuous, or no rotary embedding).
* the joint rows are, per sequence: for each kept chunk its BOS row (slot 0)
  and its kept slots ascending, then the L_q query rows -- L_j = K(1+B) + L_q
  rows, with Q from the chunk-prefill inputs and K, V from the cache.
* the joint pass is dense softmax(scale Q K^T) V over the L_j rows of each
  (sequence, head), nothing masked; its keys and values are the cache the
  decoding steps then read (prefix = the L_j joint rows, no separate static
  rows).
"""

import numpy as np


def rope_rotate_ref(x, delta, base):
    """Rotate the rotary pairs of x (..., d) by delta positions, float64.

    delta broadcasts against x's leading axes; base = 0 returns x unchanged.
    """
    x = np.asarray(x, dtype=np.float64)
    if base == 0:
        return x.copy()
    d = x.shape[-1]
    half = d // 2
    out = np.empty_like(x)
    delta = np.asarray(delta, dtype=np.float64)
    for i in range(half):
        theta = float(base) ** (-2.0 * i / d)
        ang = delta * theta
        c, s = np.cos(ang), np.sin(ang)
        a, b = x[..., i], x[..., i + half]
        out[..., i] = a * c - b * s
        out[..., i + half] = b * c + a * s
    return out


def joint_deltas(top_k, tok_budget, q_len, chunk_len):
    """Position shift of every joint row: (K(1+B) + L_q,)."""
    c1 = chunk_len + 1
    per_chunk = [k * c1 for k in range(top_k) for _ in range(1 + tok_budget)]
    return np.array(per_chunk + [(top_k - 1) * c1] * q_len, dtype=np.float64)


def joint_rows_ref(q_pre, k_cache, v_cache, q_qm, k_qm, v_qm, chunk_idx, tok_slot, q_len, base):
    """Joint Q (B, Lj, Hq, d), K and V (B, Lj, Hkv, d), float64, rotated to the joint positions.

    q_pre (B, N, 1+C, Hq, d); k_cache / v_cache (B, N, Hkv, 1+C, d); q_qm / k_qm /
    v_qm (B, Lq+Lm, H, d) shared or (B, N, Lq+Lm, H, d) per chunk (chunk 0's copy).
    """
    f = lambda a: np.asarray(a, dtype=np.float64)
    q_pre, k_cache, v_cache = f(q_pre), f(k_cache), f(v_cache)
    q_qm, k_qm, v_qm = f(q_qm), f(k_qm), f(v_qm)
    if q_qm.ndim == 5:
        q_qm, k_qm, v_qm = q_qm[:, 0], k_qm[:, 0], v_qm[:, 0]
    ci, ts = np.asarray(chunk_idx), np.asarray(tok_slot)
    bsz = q_pre.shape[0]
    top_k, tok_budget = ts.shape[1], ts.shape[2]
    qs, ks, vs = [], [], []
    for b in range(bsz):
        qr, kr, vr = [], [], []
        for kk in range(top_k):
            n = int(ci[b, kk])
            for slot in [0] + [int(x) for x in ts[b, kk]]:
                qr.append(q_pre[b, n, slot])          # (Hq, d)
                kr.append(k_cache[b, n, :, slot])     # (Hkv, d)
                vr.append(v_cache[b, n, :, slot])
        for j in range(q_len):
            qr.append(q_qm[b, j])
            kr.append(k_qm[b, j])
            vr.append(v_qm[b, j])
        qs.append(np.stack(qr))
        ks.append(np.stack(kr))
        vs.append(np.stack(vr))
    q, k, v = np.stack(qs), np.stack(ks), np.stack(vs)
    delta = joint_deltas(top_k, tok_budget, q_len, k_cache.shape[3] - 1)[None, :, None]
    return rope_rotate_ref(q, delta, base), rope_rotate_ref(k, delta, base), v


def joint_attention_ref(q, k, v, scale=None):
    """Dense bidirectional attention over the joint rows: O (B, Lj, Hq, d), natural-log LSE (B, Hq, Lj)."""
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    bsz, lj, hq, d = q.shape
    hkv = k.shape[2]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(d)
    o = np.zeros_like(q)
    lse = np.zeros((bsz, hq, lj))
    for b in range(bsz):
        for h in range(hq):
            g = h // (hq // hkv)
            s = scale * (q[b, :, h] @ k[b, :, g].T)
            m = s.max(axis=1, keepdims=True)
            ex = np.exp(s - m)
            z = ex.sum(axis=1, keepdims=True)
            o[b, :, h] = (ex / z) @ v[b, :, g]
            lse[b, h] = (m + np.log(z))[:, 0]
    return o, lse
