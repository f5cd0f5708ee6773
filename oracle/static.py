"""Static-selection mode oracle: select once, compact the kept rows, decode T steps.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper scores and selects the prefix once, before denoising (Section 5.2:
chunk selection from the pseudo-label rows; Section 5.3: the retained KV is a
static cache reused at every step).  The reading taken here (the per-step mode
of stage (b) re-selects at every step instead):

* the mean query of the selection is taken over the L_m pseudo-label rows of
  the q/m block (rows L_q .. L_q+L_m-1), not over the decode rows;
* the kept rows of every (sequence, KV head) are copied once into a
  contiguous buffer, in the order the per-step decode reads them: per kept
  chunk (ascending) its BOS row (slot 0) and then its kept slots (ascending);
* each decode step attends over [compact rows ; first n_static static rows ;
  its own L_d rows], which is exactly the per-step decode with that fixed
  selection.
"""

import numpy as np

from .select import score_select_ref


def pseudo_label_queries(q_qm, q_len):
    """Pseudo-label rows (B, Lm, Hq, d) of a q/m block, shared (B, Lq+Lm, Hq, d)
    or per chunk (B, N, Lq+Lm, Hq, d) (chunk 0's copy)."""
    q = np.asarray(q_qm)
    if q.ndim == 5:
        q = q[:, 0]
    return q[:, q_len:]


def static_select_ref(q_qm, key_mean, tok_score, top_k, tok_budget, q_len, scale=None):
    """Static selection: (chunk_idx (B, K), tok_slot (B, K, Btok), scores (B, N))."""
    return score_select_ref(pseudo_label_queries(q_qm, q_len), key_mean, tok_score, top_k, tok_budget, scale)


def gather_selected_ref(x_cache, chunk_idx, tok_slot):
    """Compact buffer (B, Hkv, K*(1+Btok), d) of the kept rows of x_cache (B, N, Hkv, 1+C, d),
    copied row by row."""
    x = np.asarray(x_cache)
    ci, ts = np.asarray(chunk_idx), np.asarray(tok_slot)
    bsz, _, hkv, _, d = x.shape
    k, bt = ts.shape[1], ts.shape[2]
    out = np.zeros((bsz, hkv, k * (1 + bt), d), dtype=x.dtype)
    for b in range(bsz):
        for g in range(hkv):
            j = 0
            for kk in range(k):
                n = int(ci[b, kk])
                out[b, g, j] = x[b, n, g, 0]
                j += 1
                for i in range(bt):
                    out[b, g, j] = x[b, n, g, int(ts[b, kk, i])]
                    j += 1
    return out


def decode_compact_unit_ref(q_dec, k_dec, v_dec, k_sel, v_sel, k_static, v_static, n_static, b, h, scale=None):
    """One (sequence b, query head h) over [compact rows ; static rows ; own rows]:
    returns (o (Ld, d), lse (Ld,)), natural-log LSE."""
    hq, hkv, d = q_dec.shape[2], k_dec.shape[2], q_dec.shape[3]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(d)
    g = h // (hq // hkv)
    f = lambda a: np.asarray(a, dtype=np.float64)
    k = np.concatenate([f(k_sel[b, g]), f(k_static[b, :n_static, g]), f(k_dec[b, :, g])], axis=0)
    v = np.concatenate([f(v_sel[b, g]), f(v_static[b, :n_static, g]), f(v_dec[b, :, g])], axis=0)
    q = f(q_dec[b, :, h])
    s = scale * (q @ k.T)
    m = s.max(axis=1, keepdims=True)
    ex = np.exp(s - m)
    z = ex.sum(axis=1, keepdims=True)
    return (ex / z) @ v, (m + np.log(z))[:, 0]


def decode_compact_ref(q_dec, k_dec, v_dec, k_sel, v_sel, k_static, v_static, n_static, scale=None):
    """Whole compact decode for small inputs: o (B, Ld, Hq, d), lse (B, Hq, Ld)."""
    bsz, ld, hq, d = q_dec.shape
    o = np.zeros((bsz, ld, hq, d))
    lse = np.zeros((bsz, hq, ld))
    for b in range(bsz):
        for h in range(hq):
            ob, lb = decode_compact_unit_ref(q_dec, k_dec, v_dec, k_sel, v_sel, k_static, v_static, n_static,
                                             b, h, scale)
            o[b, :, h, :] = ob
            lse[b, h] = lb
    return o, lse
