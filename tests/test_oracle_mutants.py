"""Plant plausible mistakes in the oracle (on the CPU) and check that a pin fails.

Each mutant replaces one oracle step through ``monkeypatch``; the test passes
only if every pin listed for it raises.
"""

import numpy as np
import pytest

import oracle.chunk_score as OCS
import oracle.decode as OD
import oracle.full_mask as OF
import oracle.prefill as OP
import oracle.select as OS
import oracle.static as OT
import oracle_checks as C


def _softmax_cols(q_rows, k_rows, scale):
    s = scale * (q_rows @ k_rows.T)
    m = s.max(axis=0, keepdims=True)
    ex = np.exp(s - m)
    z = ex.sum(axis=0, keepdims=True)
    return ex / z, (m + np.log(z))[0]


def _probs_no_scale(q_rows, k_rows, scale):
    return _orig_probs(q_rows, k_rows, 1.0)


_orig_probs = OP.chunk_probs
_orig_unit = OP.prefill_unit_ref


def _unit_one_sided(*a, **k):
    u = _orig_unit(*a, **k)
    p = u["p"]
    c1 = a[0].shape[2]
    q_len = a[9]
    u["e_head"] = p[c1:c1 + q_len, 1:c1].sum(axis=0)
    return u


def _unit_twice_first(*a, **k):
    u = _orig_unit(*a, **k)
    p = u["p"]
    c1 = a[0].shape[2]
    q_len = a[9]
    u["e_head"] = 2 * p[c1:c1 + q_len, 1:c1].sum(axis=0)
    return u


def _unit_includes_m_rows(*a, **k):
    u = _orig_unit(*a, **k)
    p = u["p"]
    c1 = a[0].shape[2]
    u["e_head"] = p[c1:, 1:c1].sum(axis=0) + p[1:c1, c1:].sum(axis=1)
    return u


def _key_mean_with_bos(k_pre):
    return np.asarray(k_pre, np.float64).mean(axis=2)


def _topk_high_index(x, k):
    x = np.asarray(x, np.float64)
    order = np.lexsort((-np.arange(x.shape[0]), -x))
    return np.sort(order[:k])


def _scores_wrong_group(q_dec, key_mean, scale=None):
    q = np.asarray(q_dec, np.float64)
    km = np.asarray(key_mean, np.float64)
    hkv = km.shape[2]
    d = q.shape[3]
    scale = 1 / np.sqrt(d) if not scale else scale
    qbar = q.mean(axis=1)
    s = np.zeros((q.shape[0], km.shape[1]))
    for h in range(q.shape[2]):
        s += scale * np.einsum("bd,bnd->bn", qbar[:, h], km[:, :, h % hkv])
    return s


def _rank_high_first_tie(tok_score):
    e = np.asarray(tok_score, np.float64)
    rank = np.zeros(e.shape, np.int32)
    for b in range(e.shape[0]):
        for n in range(e.shape[1]):
            order = np.lexsort((-np.arange(e.shape[2]), -e[b, n]))
            rank[b, n, order] = np.arange(e.shape[2])
    return rank


_orig_rows = OD.decode_kv_rows


def _rows_no_bos(x_cache, x_static, x_dec, chunk_idx, tok_slot, n_static, b, g):
    parts = [np.asarray(x_cache[b, n, g, np.asarray(tok_slot)[b, kk]], np.float64)
             for kk, n in enumerate(np.asarray(chunk_idx)[b])]
    parts.append(np.asarray(x_static[b, :n_static, g], np.float64))
    parts.append(np.asarray(x_dec[b, :, g], np.float64))
    return np.concatenate(parts)


def _rows_no_static(x_cache, x_static, x_dec, chunk_idx, tok_slot, n_static, b, g):
    return _orig_rows(x_cache, x_static, x_dec, chunk_idx, tok_slot, 0, b, g)


def _rows_slot_off_by_one(x_cache, x_static, x_dec, chunk_idx, tok_slot, n_static, b, g):
    return _orig_rows(x_cache, x_static, x_dec, chunk_idx, np.asarray(tok_slot) - 1, n_static, b, g)


def _gather_no_bos(x_cache, chunk_idx, tok_slot):
    x = np.asarray(x_cache)
    ci, ts = np.asarray(chunk_idx), np.asarray(tok_slot)
    out = []
    for b in range(x.shape[0]):
        out.append(np.stack([np.concatenate([x[b, int(n), g, ts[b, kk]] for kk, n in enumerate(ci[b])])
                             for g in range(x.shape[2])]))
    return np.stack(out)


def _unit_mass_with_bos(*a, **k):
    u = _orig_unit(*a, **k)
    c1 = a[0].shape[2]
    u["content_mass"] = u["p"][c1:, :c1].sum(axis=1)
    return u


def _unit_q2c_both(*a, **k):
    u = _orig_unit(*a, **k)
    u["e_q2c_head"] = u["e_head"]
    return u


def _score_mean_of_logs(content_mass, q_len):
    nll = -np.log(np.asarray(content_mass, np.float64))          # per head
    s_i = nll[..., :q_len].mean(axis=-1)
    s_p = nll[..., q_len:].mean(axis=-1) if nll.shape[-1] > q_len else 0 * s_i
    return (s_i + s_p).mean(axis=2)


def _score_one_normaliser(content_mass, q_len):
    a = np.asarray(content_mass, np.float64).mean(axis=2)
    return -np.log(a).mean(axis=-1)


def _score_no_pseudo_labels(content_mass, q_len):
    a = np.asarray(content_mass, np.float64).mean(axis=2)
    return -np.log(a[..., :q_len]).mean(axis=-1)


_orig_select_ranked = OCS.select_ranked_ref


def _select_ranked_ignores_order(chunk_score, tok_rank, top_k, tok_budget, lowest=True):
    return _orig_select_ranked(chunk_score, tok_rank, top_k, tok_budget, lowest=False)


_orig_rope = OF.rope_rotate_ref
_orig_joint_rows = OF.joint_rows_ref


def _rope_interleaved(x, delta, base):
    x = np.asarray(x, np.float64)
    if base == 0:
        return x.copy()
    d = x.shape[-1]
    out = np.empty_like(x)
    delta = np.asarray(delta, np.float64)
    for i in range(d // 2):
        ang = delta * float(base) ** (-2.0 * i / d)
        a, b = x[..., 2 * i], x[..., 2 * i + 1]
        out[..., 2 * i] = a * np.cos(ang) - b * np.sin(ang)
        out[..., 2 * i + 1] = b * np.cos(ang) + a * np.sin(ang)
    return out


def _rope_wrong_frequency(x, delta, base):
    x = np.asarray(x, np.float64)
    if base == 0:
        return x.copy()
    d = x.shape[-1]
    half = d // 2
    out = np.empty_like(x)
    delta = np.asarray(delta, np.float64)
    for i in range(half):
        ang = delta * float(base) ** (-1.0 * i / d)
        a, b = x[..., i], x[..., i + half]
        out[..., i] = a * np.cos(ang) - b * np.sin(ang)
        out[..., i + half] = b * np.cos(ang) + a * np.sin(ang)
    return out


def _rope_backwards(x, delta, base):
    return _orig_rope(x, -np.asarray(delta, np.float64), base)


def _deltas_query_one_chunk_late(top_k, tok_budget, q_len, chunk_len):
    c1 = chunk_len + 1
    return np.array([k * c1 for k in range(top_k) for _ in range(1 + tok_budget)] + [top_k * c1] * q_len, float)


def _joint_rows_values_rotated(*a, **k):
    q, kk, v = _orig_joint_rows(*a, **k)
    ci, ts, q_len, base = a[6], a[7], a[8], a[9]
    deltas = OF.joint_deltas(np.asarray(ts).shape[1], np.asarray(ts).shape[2], q_len, np.asarray(a[1]).shape[3] - 1)
    return q, kk, _orig_rope(v, deltas[None, :, None], base)


MUTANTS = [
    ("softmax over columns", OP, "chunk_probs", _softmax_cols,
     [C.check_prefill_golden, lambda: C.check_prefill_sdpa(3)]),
    ("scale dropped", OP, "chunk_probs", _probs_no_scale,
     [lambda: C.check_prefill_sdpa(3), lambda: C.check_prefill_blockdiag_bruteforce(1)]),
    ("Eq. 5 one-sided", OP, "prefill_unit_ref", _unit_one_sided,
     [C.check_prefill_golden, lambda: C.check_prefill_q_zero(5)]),
    ("Eq. 5 second term transposed", OP, "prefill_unit_ref", _unit_twice_first,
     [C.check_prefill_golden, lambda: C.check_prefill_blockdiag_bruteforce(1)]),
    ("Eq. 5 counts the pseudo-label rows", OP, "prefill_unit_ref", _unit_includes_m_rows,
     [C.check_prefill_golden, lambda: C.check_prefill_q_zero(5)]),
    ("key mean includes BOS", OP, "key_mean_ref", _key_mean_with_bos,
     [C.check_prefill_golden, lambda: C.check_key_mean_const(9)]),
    ("ties to the higher index", OS, "topk_ref", _topk_high_index,
     [C.check_select_golden, lambda: C.check_topk_bruteforce(13)]),
    ("token ranks break ties to the higher index", OS, "token_rank_ref", _rank_high_first_tie,
     [C.check_select_golden, lambda: C.check_token_rank(16)]),
    ("query head mapped to the wrong KV head", OS, "chunk_scores_ref", _scores_wrong_group,
     [lambda: C.check_chunk_score_gqa_groups(12)]),
    ("decode drops the chunk BOS rows", OD, "decode_kv_rows", _rows_no_bos,
     [C.check_decode_golden, lambda: C.check_decode_dense(14)]),
    ("decode drops the static rows", OD, "decode_kv_rows", _rows_no_static,
     [C.check_decode_golden, lambda: C.check_decode_dense(14)]),
    ("decode slot off by one", OD, "decode_kv_rows", _rows_slot_off_by_one,
     [C.check_decode_golden]),
    ("static selection averages every q/m row", OT, "pseudo_label_queries", lambda q_qm, q_len: np.asarray(q_qm),
     [C.check_static_golden]),
    ("static selection uses the query rows", OT, "pseudo_label_queries",
     lambda q_qm, q_len: np.asarray(q_qm)[:, :q_len], [C.check_static_golden]),
    ("gather drops the chunk BOS rows", OT, "gather_selected_ref", _gather_no_bos,
     [C.check_static_golden, lambda: C.check_gather_matches_decode_rows(1),
      lambda: C.check_compact_decode_equals_gathered(7, 3)]),
    ("content mass includes the BOS column", OP, "prefill_unit_ref", _unit_mass_with_bos,
     [C.check_prefill_golden, C.check_chunk_score_golden, lambda: C.check_chunk_score_uniform(21, 4),
      lambda: C.check_chunk_score_bruteforce(22)]),
    ("query-to-chunk score keeps both sums", OP, "prefill_unit_ref", _unit_q2c_both,
     [C.check_prefill_golden, C.check_chunk_score_golden]),
    ("chunk score averages the logs over heads", OCS, "prefill_chunk_score_ref", _score_mean_of_logs,
     [C.check_chunk_score_golden, lambda: C.check_chunk_score_bruteforce(22)]),
    ("chunk score uses one length for both terms", OCS, "prefill_chunk_score_ref", _score_one_normaliser,
     [C.check_prefill_golden, C.check_chunk_score_golden, lambda: C.check_chunk_score_uniform(21, 4)]),
    ("chunk score drops the pseudo-label term", OCS, "prefill_chunk_score_ref", _score_no_pseudo_labels,
     [C.check_prefill_golden, C.check_chunk_score_golden, lambda: C.check_chunk_score_uniform(21, 4)]),
    ("selection keeps the highest scores", OCS, "select_ranked_ref", _select_ranked_ignores_order,
     [C.check_chunk_score_golden, lambda: C.check_select_ranked_bruteforce(24)]),
    ("rotary pairs interleaved", OF, "rope_rotate_ref", _rope_interleaved,
     [C.check_full_mask_golden, lambda: C.check_rope_composition(31), lambda: C.check_joint_rows(32)]),
    ("rotary frequency exponent halved", OF, "rope_rotate_ref", _rope_wrong_frequency,
     [C.check_full_mask_golden, lambda: C.check_rope_composition(31)]),
    ("rows moved backwards", OF, "rope_rotate_ref", _rope_backwards,
     [C.check_full_mask_golden, lambda: C.check_rope_composition(31), lambda: C.check_joint_rows(32)]),
    ("query rows placed one chunk late", OF, "joint_deltas", _deltas_query_one_chunk_late,
     [C.check_full_mask_golden]),
    ("values rotated with the keys", OF, "joint_rows_ref", _joint_rows_values_rotated,
     [lambda: C.check_joint_rows(32)]),
]


@pytest.mark.parametrize("name,mod,attr,repl,checks", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(monkeypatch, name, mod, attr, repl, checks):
    monkeypatch.setattr(mod, attr, repl)
    for chk in checks:
        with pytest.raises(Exception):
            chk()
