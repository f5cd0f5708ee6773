"""Stage (c) oracle: sparse decode attention at one denoising step.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Section 5.3 ("Prefix Reuse"): the retained KV of the selected chunks and the
query KV form a static cache reused at every step; at each step only the
response block is processed, its KV concatenated with that cache, and the
attention is bidirectional.  The KV rows of one (sequence, KV head) are, in
order:

  for each selected chunk (ascending): its BOS row (slot 0), then the rows at
  its kept slots (ascending);
  the first n_static rows of the static query KV (the L_q query rows);
  the L_d rows of the decode block itself.

The order does not change the result (attention is invariant to permuting KV
rows); it is fixed only so that the row list is well defined.

Layouts: q_dec (B, Ld, Hq, d); k_dec / v_dec (B, Ld, Hkv, d);
k_cache / v_cache (B, N, Hkv, 1+C, d); k_static / v_static (B, Ls, Hkv, d)
with Ls >= n_static; chunk_idx (B, K); tok_slot (B, K, Btok).
"""

import numpy as np


def decode_kv_rows(x_cache, x_static, x_dec, chunk_idx, tok_slot, n_static, b, g):
    """KV rows (L_kv, d) float64 seen by the decode block of sequence b, KV head g."""
    parts = []
    for kk, n in enumerate(np.asarray(chunk_idx)[b]):
        parts.append(np.asarray(x_cache[b, n, g, 0:1], dtype=np.float64))
        parts.append(np.asarray(x_cache[b, n, g, np.asarray(tok_slot)[b, kk]], dtype=np.float64))
    parts.append(np.asarray(x_static[b, :n_static, g], dtype=np.float64))
    parts.append(np.asarray(x_dec[b, :, g], dtype=np.float64))
    return np.concatenate(parts, axis=0)


def decode_unit_ref(q_dec, k_dec, v_dec, k_cache, v_cache, chunk_idx, tok_slot,
                    k_static, v_static, n_static, b, h, scale=None):
    """One (sequence b, query head h): returns (o (Ld, d), lse (Ld,)), natural-log LSE."""
    hq, hkv, d = q_dec.shape[2], k_dec.shape[2], q_dec.shape[3]
    if scale is None or scale == 0:
        scale = 1.0 / np.sqrt(d)
    g = h // (hq // hkv)
    q = np.asarray(q_dec[b, :, h], dtype=np.float64)
    k = decode_kv_rows(k_cache, k_static, k_dec, chunk_idx, tok_slot, n_static, b, g)
    v = decode_kv_rows(v_cache, v_static, v_dec, chunk_idx, tok_slot, n_static, b, g)
    s = scale * (q @ k.T)
    m = s.max(axis=1, keepdims=True)
    ex = np.exp(s - m)
    z = ex.sum(axis=1, keepdims=True)
    o = (ex / z) @ v
    return o, (m + np.log(z))[:, 0]


def decode_ref(q_dec, k_dec, v_dec, k_cache, v_cache, chunk_idx, tok_slot,
               k_static, v_static, n_static, scale=None):
    """Whole stage (c) for small inputs: o (B, Ld, Hq, d), lse (B, Hq, Ld)."""
    bsz, ld, hq, d = q_dec.shape
    o = np.zeros((bsz, ld, hq, d))
    lse = np.zeros((bsz, hq, ld))
    for b in range(bsz):
        for h in range(hq):
            ob, lb = decode_unit_ref(q_dec, k_dec, v_dec, k_cache, v_cache, chunk_idx,
                                     tok_slot, k_static, v_static, n_static, b, h, scale)
            o[b, :, h, :] = ob
            lse[b, h] = lb
    return o, lse
