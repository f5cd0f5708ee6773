"""Pins for the oracle: each check compares it with something other than itself.

Every check reaches the oracle through its submodules at call time
(``oracle.prefill.prefill_ref`` ...), so the mutation tests can plant a
mistake in one oracle step with ``monkeypatch`` and confirm that some check
fails.  Pins used:

* hand-derived worked examples (``tests/golden/*.json``; the paper prints no
  numeric example, so each fixture derives its values from the definitions);
* brute force: the N chunk sequences concatenated with an explicit
  block-diagonal -inf mask and a dense softmax (scipy); subset enumeration for
  top-K;
* library routines: torch scaled_dot_product_attention in float64 on the CPU,
  numpy stable argsort;
* closed forms: Q = 0, V = constant, constant content keys;
* invariants: probability rows sum to one, KV-row permutation invariance.
"""

import itertools
import json
import os
from fractions import Fraction

import numpy as np
import scipy.special
import torch

import oracle.chunk_score as OCS
import oracle.decode as OD
import oracle.full_mask as OF
import oracle.prefill as OP
import oracle.select as OS
import oracle.static as OT

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _frac(x):
    return float(Fraction(x))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def tiny_prefill_inputs(seed, B=2, N=3, C=5, Lq=2, Lm=3, Hq=4, Hkv=2, d=8, per_chunk=False):
    rng = np.random.default_rng(seed)
    qm_shape = (B, N, Lq + Lm) if per_chunk else (B, Lq + Lm)
    return {
        "q_pre": rng.standard_normal((B, N, 1 + C, Hq, d)),
        "k_pre": rng.standard_normal((B, N, 1 + C, Hkv, d)),
        "v_pre": rng.standard_normal((B, N, 1 + C, Hkv, d)),
        "q_qm": rng.standard_normal(qm_shape + (Hq, d)),
        "k_qm": rng.standard_normal(qm_shape + (Hkv, d)),
        "v_qm": rng.standard_normal(qm_shape + (Hkv, d)),
    }


def _prefill(x, Lq, scale=None):
    return OP.prefill_ref(x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"], Lq, scale)


# ----------------------------------------------------------------------------- stage (a)

def check_prefill_golden():
    g = _load("prefill_worked_example.json")
    x = {k: np.array(g[k], dtype=np.float64) for k in ("q_pre", "k_pre", "v_pre", "q_qm", "k_qm", "v_qm")}
    r = _prefill(x, g["dims"]["L_q"], g["dims"]["scale"])
    want_o = np.array([[_frac(v) for v in row] for row in g["expect_o_rows"]])
    np.testing.assert_allclose(r["o"][0, 0, :, 0, :], want_o, rtol=0, atol=1e-12)
    want_e = np.array([_frac(v) for v in g["expect_tok_score"]])
    np.testing.assert_allclose(r["tok_score"][0, 0], want_e, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["lse"][0, 0, 0], np.log(np.array(g["expect_lse_of"], float)), atol=1e-12)
    np.testing.assert_allclose(r["key_mean"][0, 0, 0], g["expect_key_mean"], atol=1e-15)
    u = OP.prefill_unit_ref(x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"],
                            0, 0, 0, g["dims"]["L_q"], g["dims"]["scale"])
    want_p = np.array([[_frac(v) for v in row] for row in g["expect_probs"]])
    np.testing.assert_allclose(u["p"], want_p, rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["content_mass"][0, 0, 0], [_frac(v) for v in g["expect_content_mass"]], atol=1e-12)
    np.testing.assert_allclose(r["tok_score_q2c"][0, 0], [_frac(v) for v in g["expect_tok_score_q2c"]], atol=1e-12)
    np.testing.assert_allclose(OCS.prefill_chunk_score_ref(r["content_mass"], g["dims"]["L_q"])[0, 0],
                               np.log(_frac(g["expect_chunk_score_exp"])), atol=1e-12)


def check_prefill_blockdiag_bruteforce(seed, per_chunk=False):
    """Concatenate the N chunk sequences of each (b, h), mask across chunks with -inf,
    take one dense softmax and compare O, LSE and the Eq. 5 score (explicit loops)."""
    B, N, C, Lq, Lm, Hq, Hkv, d = 2, 3, 5, 2, 3, 4, 2, 8
    x = tiny_prefill_inputs(seed, B, N, C, Lq, Lm, Hq, Hkv, d, per_chunk)
    scale = 1.0 / np.sqrt(d)
    r = _prefill(x, Lq)
    sc = 1 + C + Lq + Lm
    tot = N * sc
    for b in range(B):
        e_bf = np.zeros((N, C))
        for h in range(Hq):
            g = h // (Hq // Hkv)
            Q = np.zeros((tot, d))
            K = np.zeros((tot, d))
            V = np.zeros((tot, d))
            owner = np.zeros(tot, dtype=int)
            for n in range(N):
                for s in range(sc):
                    row = n * sc + s
                    owner[row] = n
                    if s <= C:
                        Q[row], K[row], V[row] = x["q_pre"][b, n, s, h], x["k_pre"][b, n, s, g], x["v_pre"][b, n, s, g]
                    else:
                        j = s - 1 - C
                        src = (lambda t: t[b, n, j]) if per_chunk else (lambda t: t[b, j])
                        Q[row], K[row], V[row] = src(x["q_qm"])[h], src(x["k_qm"])[g], src(x["v_qm"])[g]
            mask = np.where(owner[:, None] == owner[None, :], 0.0, -np.inf)
            S = scale * Q @ K.T + mask
            P = scipy.special.softmax(S, axis=1)
            O = P @ V
            lse = scipy.special.logsumexp(S, axis=1)
            for n in range(N):
                rows = slice(n * sc, (n + 1) * sc)
                np.testing.assert_allclose(r["o"][b, n, :, h, :], O[rows], rtol=0, atol=1e-12)
                np.testing.assert_allclose(r["lse"][b, n, h], lse[rows], rtol=0, atol=1e-12)
                for j in range(C):
                    cj = n * sc + 1 + j
                    for k in range(Lq):
                        qk = n * sc + 1 + C + k
                        e_bf[n, j] += P[qk, cj] + P[cj, qk]
        np.testing.assert_allclose(r["tok_score"][b], e_bf, rtol=0, atol=1e-12)


def check_prefill_sdpa(seed):
    """Per-chunk O against torch's scaled_dot_product_attention (float64, CPU)."""
    B, N, C, Lq, Lm, Hq, Hkv, d = 1, 2, 9, 3, 4, 6, 2, 16
    x = tiny_prefill_inputs(seed, B, N, C, Lq, Lm, Hq, Hkv, d)
    r = _prefill(x, Lq)
    for b in range(B):
        for n in range(N):
            q = np.concatenate([x["q_pre"][b, n], x["q_qm"][b]], axis=0)       # (Sc, Hq, d)
            k = np.concatenate([x["k_pre"][b, n], x["k_qm"][b]], axis=0)
            v = np.concatenate([x["v_pre"][b, n], x["v_qm"][b]], axis=0)
            rep = Hq // Hkv
            qt = torch.from_numpy(q).permute(1, 0, 2)
            kt = torch.from_numpy(np.repeat(k, rep, axis=1)).permute(1, 0, 2)
            vt = torch.from_numpy(np.repeat(v, rep, axis=1)).permute(1, 0, 2)
            ot = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt).permute(1, 0, 2).numpy()
            np.testing.assert_allclose(r["o"][b, n], ot, rtol=0, atol=1e-12)


def check_prefill_q_zero(seed):
    """Q = 0: every probability is 1/S_c, O is the mean of the V rows, e_j = 2 Hq Lq / S_c."""
    B, N, C, Lq, Lm, Hq, Hkv, d = 1, 2, 6, 3, 2, 4, 1, 8
    x = tiny_prefill_inputs(seed, B, N, C, Lq, Lm, Hq, Hkv, d)
    x["q_pre"][:] = 0
    x["q_qm"][:] = 0
    r = _prefill(x, Lq)
    sc = 1 + C + Lq + Lm
    for n in range(N):
        vrows = np.concatenate([x["v_pre"][0, n, :, 0], x["v_qm"][0, :, 0]], axis=0)
        for h in range(Hq):
            np.testing.assert_allclose(r["o"][0, n, :, h], np.broadcast_to(vrows.mean(axis=0), (sc, d)), atol=1e-12)
        np.testing.assert_allclose(r["lse"][0, n], np.log(sc), atol=1e-12)
    np.testing.assert_allclose(r["tok_score"], 2.0 * Hq * Lq / sc, atol=1e-12)


def check_prefill_v_const(seed):
    """V rows all equal to one vector v: O = v in every row and head."""
    x = tiny_prefill_inputs(seed)
    v = np.arange(x["v_pre"].shape[-1], dtype=np.float64) - 3.5
    x["v_pre"][:] = v
    x["v_qm"][:] = v
    r = _prefill(x, 2)
    np.testing.assert_allclose(r["o"], np.broadcast_to(v, r["o"].shape), atol=1e-12)


def check_prefill_rowsums(seed):
    """Every probability row is non-negative and sums to one."""
    x = tiny_prefill_inputs(seed)
    for (b, n, h) in [(0, 0, 0), (1, 2, 3), (0, 1, 2)]:
        u = OP.prefill_unit_ref(x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"], b, n, h, 2)
        assert (u["p"] >= 0).all()
        np.testing.assert_allclose(u["p"].sum(axis=1), 1.0, atol=1e-12)


def check_cache_exact(seed):
    """The cache is the chunk's BOS + content rows, bit for bit, at [b][n][g][slot]."""
    x = tiny_prefill_inputs(seed)
    kp = x["k_pre"].astype(np.float32)
    kc = OP.cache_ref(kp)
    assert kc.dtype == np.float32
    B, N, C1, Hkv, d = kp.shape
    for b, n, g, s in itertools.product(range(B), range(N), range(Hkv), range(C1)):
        assert np.array_equal(kc[b, n, g, s], kp[b, n, s, g])


def check_key_mean_const(seed):
    """Content keys equal to one vector per (b, n, g) and a random BOS row: the mean is that vector."""
    x = tiny_prefill_inputs(seed)
    k = x["k_pre"].copy()
    B, N, C1, Hkv, d = k.shape
    const = np.random.default_rng(seed + 1).standard_normal((B, N, Hkv, d))
    k[:, :, 1:] = const[:, :, None]
    np.testing.assert_allclose(OP.key_mean_ref(k), const, atol=1e-14)


# ----------------------------------------------------------------------------- stage (b)

def check_select_golden():
    g = _load("select_worked_example.json")
    q = np.array(g["q_dec"], float)
    km = np.array(g["key_mean"], float)
    ts = np.array(g["tok_score"], float)
    s = OS.chunk_scores_ref(q, km, g["dims"]["scale"])
    np.testing.assert_allclose(s[0], g["expect_scores"], atol=1e-12)
    rank = OS.token_rank_ref(ts)
    assert rank.tolist() == g["expect_tok_rank"]
    for case in g["cases"]:
        ci, tsl, _ = OS.score_select_ref(q, km, ts, case["top_k"], case["tok_budget"], g["dims"]["scale"])
        assert ci[0].tolist() == case["chunk_idx"], case
        assert tsl[0].tolist() == case["tok_slot"], case
        assert OS.tokens_by_rank_ref(rank, ci, case["tok_budget"])[0].tolist() == case["tok_slot"], case


def check_chunk_score_zero_query(seed):
    """Q_dec = 0: all scores 0, so the first K chunks are kept (ties to the lower index)."""
    rng = np.random.default_rng(seed)
    q = np.zeros((2, 5, 4, 8))
    km = rng.standard_normal((2, 7, 2, 8))
    e = rng.standard_normal((2, 7, 6))
    ci, _, s = OS.score_select_ref(q, km, e, 3, 2)
    assert np.all(s == 0)
    assert ci.tolist() == [[0, 1, 2], [0, 1, 2]]


def check_chunk_score_linear(seed):
    """The score is linear in the decode queries: 2 Q_dec -> 2 s; Q1 + Q2 -> s1 + s2."""
    rng = np.random.default_rng(seed)
    q1, q2 = rng.standard_normal((2, 1, 6, 4, 8))
    km = rng.standard_normal((1, 5, 2, 8))
    s1 = OS.chunk_scores_ref(q1, km)
    s2 = OS.chunk_scores_ref(q2, km)
    np.testing.assert_allclose(OS.chunk_scores_ref(2 * q1, km), 2 * s1, atol=1e-12)
    np.testing.assert_allclose(OS.chunk_scores_ref(q1 + q2, km), s1 + s2, atol=1e-12)


def check_chunk_score_gqa_groups(seed):
    """Query head h reads KV head h // (Hq/Hkv): queries only in heads 2, 3 (group 1) and key
    means only in KV head 0 give all-zero scores; key means in KV head 1 give non-zero ones."""
    rng = np.random.default_rng(seed)
    q = np.zeros((1, 3, 4, 8))
    q[:, :, 2:] = rng.standard_normal((1, 3, 2, 8))
    km = np.zeros((1, 4, 2, 8))
    km[:, :, 0] = rng.standard_normal((1, 4, 8))
    assert np.all(OS.chunk_scores_ref(q, km) == 0)
    km2 = np.zeros((1, 4, 2, 8))
    km2[:, :, 1] = rng.standard_normal((1, 4, 8))
    assert np.all(OS.chunk_scores_ref(q, km2) != 0)


def check_topk_bruteforce(seed):
    """Among all size-k subsets exactly one has every member ranking above every
    non-member (score descending, index ascending); it is the oracle's answer."""
    rng = np.random.default_rng(seed)
    for trial in range(30):
        n = int(rng.integers(1, 8))
        x = rng.integers(-3, 4, size=n).astype(np.float64)      # many ties
        for k in range(1, n + 1):
            def beats(i, j):
                return x[i] > x[j] or (x[i] == x[j] and i < j)
            good = [set(c) for c in itertools.combinations(range(n), k)
                    if all(beats(i, j) for i in c for j in range(n) if j not in c)]
            assert len(good) == 1
            got = OS.topk_ref(x, k)
            assert set(got.tolist()) == good[0]
            assert list(got) == sorted(got)
            stable = np.sort(np.argsort(-x, kind="stable")[:k])
            assert np.array_equal(got, stable)


def check_token_rank(seed):
    """Ranks against a library routine (numpy stable argsort of -e) and, on small
    integer scores with many ties, against counting: rank_j = #{i: e_i > e_j or
    (e_i = e_j and i < j)}; selecting ranks below B reproduces the top-B slots."""
    rng = np.random.default_rng(seed)
    e = rng.integers(0, 4, size=(2, 3, 9)).astype(np.float64)
    r = OS.token_rank_ref(e)
    for b in range(2):
        for n in range(3):
            cnt = [sum(1 for i in range(9) if e[b, n, i] > e[b, n, j] or (e[b, n, i] == e[b, n, j] and i < j))
                   for j in range(9)]
            assert r[b, n].tolist() == cnt
            inv = np.empty(9, dtype=np.int64)
            inv[np.argsort(-e[b, n], kind="stable")] = np.arange(9)
            assert np.array_equal(r[b, n], inv)
    ci = np.array([[0, 2], [1, 2]])
    for bt in (1, 4, 9):
        want = np.stack([np.stack([1 + OS.topk_ref(e[b, n], bt) for n in ci[b]]) for b in range(2)])
        assert np.array_equal(OS.tokens_by_rank_ref(r, ci, bt), want)


# ----------------------------------------------------------------------------- prefill-time chunk score

def check_chunk_score_golden():
    """Two heads with different content masses (head average before the log), and
    selection of the K lowest / highest given scores with a tie."""
    g = _load("chunk_score_worked_example.json")
    x = {k: np.array(g[k], dtype=np.float64) for k in ("q_pre", "k_pre", "v_pre", "q_qm", "k_qm", "v_qm")}
    r = _prefill(x, g["dims"]["L_q"], g["dims"]["scale"])
    want_mass = np.array([[_frac(v) for v in row] for row in g["expect_content_mass"]])
    np.testing.assert_allclose(r["content_mass"][0, 0], want_mass, atol=1e-12)
    np.testing.assert_allclose(r["tok_score"][0, 0], [_frac(v) for v in g["expect_tok_score"]], atol=1e-12)
    np.testing.assert_allclose(r["tok_score_q2c"][0, 0], [_frac(v) for v in g["expect_tok_score_q2c"]], atol=1e-12)
    s = OCS.prefill_chunk_score_ref(r["content_mass"], g["dims"]["L_q"])
    np.testing.assert_allclose(s[0, 0], np.log(_frac(g["expect_chunk_score_exp"])), atol=1e-12)
    sel = g["select"]
    for case in sel["cases"]:
        ci, ts = OCS.select_ranked_ref(np.array(sel["chunk_score"], float), np.array(sel["tok_rank"]),
                                       case["top_k"], sel["tok_budget"], bool(case["lowest"]))
        assert ci.tolist() == case["chunk_idx"], case
        assert ts.tolist() == case["tok_slot"], case


def check_chunk_score_uniform(seed, m_len):
    """All queries zero: every row is uniform over the S_c columns, so each q/m row
    puts C/S_c on the content and s = -ln(C/S_c) per non-empty term."""
    x = tiny_prefill_inputs(seed, Lq=3, Lm=m_len, C=7)
    x["q_pre"][:] = 0
    x["q_qm"][:] = 0
    r = _prefill(x, 3)
    sc = 1 + 7 + 3 + m_len
    np.testing.assert_allclose(r["content_mass"], 7 / sc, atol=1e-13)
    terms = 2 if m_len > 0 else 1
    np.testing.assert_allclose(OCS.prefill_chunk_score_ref(r["content_mass"], 3), -terms * np.log(7 / sc),
                               atol=1e-12)


def check_chunk_score_bruteforce(seed):
    """Against the dense block-diagonal forward of all chunks at once (scipy
    softmax over the concatenated sequences with -inf across chunks): the mass of
    every q/m row on its own chunk's content columns, then the score written out
    row by row with explicit loops."""
    B, N, C, Lq, Lm, Hq, Hkv, d = 1, 3, 5, 2, 3, 4, 2, 8
    x = tiny_prefill_inputs(seed, B, N, C, Lq, Lm, Hq, Hkv, d)
    r = _prefill(x, Lq)
    sc = 1 + C + Lq + Lm
    scale = 1 / np.sqrt(d)
    for h in range(Hq):
        g = h // (Hq // Hkv)
        qs = np.concatenate([np.concatenate([x["q_pre"][0, n, :, h], x["q_qm"][0, :, h]]) for n in range(N)])
        ks = np.concatenate([np.concatenate([x["k_pre"][0, n, :, g], x["k_qm"][0, :, g]]) for n in range(N)])
        logits = scale * qs @ ks.T
        for n in range(N):
            for m in range(N):
                if m != n:
                    logits[n * sc:(n + 1) * sc, m * sc:(m + 1) * sc] = -np.inf
        p = scipy.special.softmax(logits, axis=1)
        for n in range(N):
            for i in range(Lq + Lm):
                row = n * sc + 1 + C + i
                np.testing.assert_allclose(r["content_mass"][0, n, h, i], p[row, n * sc + 1:n * sc + 1 + C].sum(),
                                           atol=1e-13)
    got = OCS.prefill_chunk_score_ref(r["content_mass"], Lq)
    for n in range(N):
        want = 0.0
        for i in range(Lq + Lm):
            a = sum(r["content_mass"][0, n, h, i] for h in range(Hq)) / Hq
            want -= np.log(a) / (Lq if i < Lq else Lm)
        np.testing.assert_allclose(got[0, n], want, atol=1e-12)


def check_select_ranked_bruteforce(seed):
    """Among all size-k subsets exactly one has every member ranking before every
    non-member (score ascending, index ascending); selection of the K lowest returns
    it, and the K highest is the K lowest of the negated scores."""
    rng = np.random.default_rng(seed)
    for trial in range(20):
        n = int(rng.integers(1, 7))
        x = rng.integers(-2, 3, size=(1, n)).astype(np.float64)
        rank = np.stack([rng.permutation(4) for _ in range(n)])[None]
        for k in range(1, n + 1):
            def before(i, j):
                return x[0, i] < x[0, j] or (x[0, i] == x[0, j] and i < j)
            good = [c for c in itertools.combinations(range(n), k)
                    if all(before(i, j) for i in c for j in range(n) if j not in c)]
            assert len(good) == 1
            ci, ts = OCS.select_ranked_ref(x, rank, k, 2, lowest=True)
            assert ci[0].tolist() == list(good[0])
            for kk, c in enumerate(good[0]):
                assert ts[0, kk].tolist() == [1 + j for j in range(4) if rank[0, c, j] < 2]
            hi, _ = OCS.select_ranked_ref(-x, rank, k, 2, lowest=False)
            assert np.array_equal(hi, ci)


# ----------------------------------------------------------------------------- full-mask construction

def _mathexpr(e):
    import math
    return float(eval(e, {"__builtins__": {}}, {"sin": math.sin, "cos": math.cos}))


def check_full_mask_golden():
    g = _load("full_mask_worked_example.json")
    for case in g["rope"]:
        got = OF.rope_rotate_ref(np.array(case["x"], float), case["delta"], case["base"])
        np.testing.assert_allclose(got, [_mathexpr(e) for e in case["expect"]], atol=1e-14)
    dl = g["deltas"]
    assert OF.joint_deltas(dl["K"], dl["B"], dl["L_q"], dl["C"]).tolist() == dl["expect"]


def _rope_complex(u, pos, base):
    """Rotary embedding of u at absolute position pos, as complex multiplication of the
    rotate-half pairs (u_i + i u_{i+d/2}) by exp(i pos theta_i)."""
    d = u.shape[-1]
    half = d // 2
    theta = float(base) ** (-2.0 * np.arange(half) / d)
    z = (u[..., :half] + 1j * u[..., half:]) * np.exp(1j * np.asarray(pos, float)[..., None] * theta)
    return np.concatenate([z.real, z.imag], axis=-1)


def check_rope_composition(seed):
    """Re-rotating a row embedded at its chunk-local position p by delta equals embedding
    it at p + delta directly; moving by delta then by -delta is the identity; a common
    move leaves every q.k unchanged (scores see relative positions only)."""
    rng = np.random.default_rng(seed)
    u = rng.standard_normal((5, 16))
    p = rng.integers(0, 50, size=5)
    delta = rng.integers(0, 5000, size=5)
    for base in (10000.0, 1e6):
        local = _rope_complex(u, p, base)
        np.testing.assert_allclose(OF.rope_rotate_ref(local, delta, base), _rope_complex(u, p + delta, base),
                                   atol=1e-9)
        np.testing.assert_allclose(OF.rope_rotate_ref(OF.rope_rotate_ref(local, delta, base), -delta, base), local,
                                   atol=1e-9)
        q = rng.standard_normal(16)
        k = rng.standard_normal(16)
        np.testing.assert_allclose(OF.rope_rotate_ref(q, 1234, base) @ OF.rope_rotate_ref(k, 1234, base), q @ k,
                                   atol=1e-10)
    assert np.array_equal(OF.rope_rotate_ref(u, delta, 0), u)


def _tiny_full_mask(seed, B=2, N=4, C=6, Lq=3, Lm=2, Hq=4, Hkv=2, d=8, K=2, Bt=3):
    x = tiny_prefill_inputs(seed, B, N, C, Lq, Lm, Hq, Hkv, d)
    ci, ts = _tiny_selection(seed + 1, B, N, C, K, Bt)
    kc = OP.cache_ref(x["k_pre"])
    vc = OP.cache_ref(x["v_pre"])
    return x, kc, vc, ci, ts


def check_joint_rows(seed):
    """Joint rows without rotation: the kept cache rows in decode order (the same rows
    the static-mode gather copies), then the query rows; with rotation the values stay
    put and Q, K move by the per-row deltas."""
    x, kc, vc, ci, ts = _tiny_full_mask(seed)
    Lq = 3
    q, k, v = OF.joint_rows_ref(x["q_pre"], kc, vc, x["q_qm"], x["k_qm"], x["v_qm"], ci, ts, Lq, 0)
    n_sel = ci.shape[1] * (1 + ts.shape[2])
    np.testing.assert_array_equal(np.transpose(k[:, :n_sel], (0, 2, 1, 3)), OT.gather_selected_ref(kc, ci, ts))
    np.testing.assert_array_equal(np.transpose(v[:, :n_sel], (0, 2, 1, 3)), OT.gather_selected_ref(vc, ci, ts))
    np.testing.assert_array_equal(k[:, n_sel:], x["k_qm"][:, :Lq])
    for b in range(2):
        for kk in range(ci.shape[1]):
            n = ci[b, kk]
            np.testing.assert_array_equal(q[b, kk * (1 + ts.shape[2])], x["q_pre"][b, n, 0])
    q2, k2, v2 = OF.joint_rows_ref(x["q_pre"], kc, vc, x["q_qm"], x["k_qm"], x["v_qm"], ci, ts, Lq, 10000.0)
    np.testing.assert_array_equal(v2, v)
    deltas = OF.joint_deltas(ci.shape[1], ts.shape[2], Lq, 6)
    np.testing.assert_allclose(k2, _rope_complex_moved(k, deltas), atol=1e-9)
    np.testing.assert_allclose(q2, _rope_complex_moved(q, deltas), atol=1e-9)


def _rope_complex_moved(x, deltas, base=10000.0):
    """Move rows (B, L, H, d) by deltas (L,) with the complex-number rotation."""
    d = x.shape[-1]
    half = d // 2
    theta = base ** (-2.0 * np.arange(half) / d)
    z = (x[..., :half] + 1j * x[..., half:]) * np.exp(1j * deltas[None, :, None, None] * theta)
    return np.concatenate([z.real, z.imag], axis=-1)


def check_joint_attention_sdpa(seed):
    """The joint pass against torch scaled_dot_product_attention (float64, CPU, no mask)."""
    x, kc, vc, ci, ts = _tiny_full_mask(seed)
    q, k, v = OF.joint_rows_ref(x["q_pre"], kc, vc, x["q_qm"], x["k_qm"], x["v_qm"], ci, ts, 3, 10000.0)
    o, lse = OF.joint_attention_ref(q, k, v)
    G = q.shape[2] // k.shape[2]
    qt = torch.from_numpy(q).permute(0, 2, 1, 3)
    kt = torch.from_numpy(np.repeat(k, G, axis=2)).permute(0, 2, 1, 3).contiguous()
    vt = torch.from_numpy(np.repeat(v, G, axis=2)).permute(0, 2, 1, 3).contiguous()
    want = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt).permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(o, want, atol=1e-12)
    s = torch.einsum("bhqd,bhkd->bhqk", qt, kt) / np.sqrt(q.shape[-1])
    np.testing.assert_allclose(lse, torch.logsumexp(s, dim=-1).numpy(), atol=1e-12)


def check_full_mask_dense(seed):
    """Everything kept (K = N, B = C) and no rotation: the joint pass is dense attention
    over all chunk rows (BOS included) followed by the query rows, built here by explicit
    concatenation."""
    B, N, C, Lq, Hq, Hkv, d = 1, 3, 4, 2, 2, 1, 8
    x = tiny_prefill_inputs(seed, B, N, C, Lq, 1, Hq, Hkv, d)
    ci = np.arange(N)[None]
    ts = np.tile(np.arange(1, C + 1), (1, N, 1))
    q, k, v = OF.joint_rows_ref(x["q_pre"], OP.cache_ref(x["k_pre"]), OP.cache_ref(x["v_pre"]), x["q_qm"], x["k_qm"],
                                x["v_qm"], ci, ts, Lq, 0)
    o, _ = OF.joint_attention_ref(q, k, v)
    for h in range(Hq):
        qa = np.concatenate([x["q_pre"][0, n, :, h] for n in range(N)] + [x["q_qm"][0, :Lq, h]])
        ka = np.concatenate([x["k_pre"][0, n, :, 0] for n in range(N)] + [x["k_qm"][0, :Lq, 0]])
        va = np.concatenate([x["v_pre"][0, n, :, 0] for n in range(N)] + [x["v_qm"][0, :Lq, 0]])
        p = scipy.special.softmax(qa @ ka.T / np.sqrt(d), axis=1)
        np.testing.assert_allclose(o[0, :, h], p @ va, atol=1e-12)


# ----------------------------------------------------------------------------- stage (c)

def check_decode_golden():
    g = _load("decode_worked_example.json")
    a = {k: np.array(g[k], float) for k in ("q_dec", "k_dec", "v_dec", "k_cache", "v_cache", "k_static", "v_static")}
    ci = np.array(g["chunk_idx"], np.int32)
    ts = np.array(g["tok_slot"], np.int32)
    o, lse = OD.decode_ref(a["q_dec"], a["k_dec"], a["v_dec"], a["k_cache"], a["v_cache"], ci, ts,
                           a["k_static"], a["v_static"], g["dims"]["n_static"], g["dims"]["scale"])
    np.testing.assert_allclose(o[0, 0, 0], [_frac(v) for v in g["expect_o"]], atol=1e-12)
    np.testing.assert_allclose(lse[0, 0, 0], np.log(g["expect_lse_of"]), atol=1e-12)


def tiny_decode_inputs(seed, B=2, N=4, C=6, Ld=3, Ls=4, Hq=4, Hkv=2, d=8):
    rng = np.random.default_rng(seed)
    return {
        "q_dec": rng.standard_normal((B, Ld, Hq, d)),
        "k_dec": rng.standard_normal((B, Ld, Hkv, d)),
        "v_dec": rng.standard_normal((B, Ld, Hkv, d)),
        "k_cache": rng.standard_normal((B, N, Hkv, 1 + C, d)),
        "v_cache": rng.standard_normal((B, N, Hkv, 1 + C, d)),
        "k_static": rng.standard_normal((B, Ls, Hkv, d)),
        "v_static": rng.standard_normal((B, Ls, Hkv, d)),
    }


def _decode(x, ci, ts, n_static):
    return OD.decode_ref(x["q_dec"], x["k_dec"], x["v_dec"], x["k_cache"], x["v_cache"], ci, ts,
                         x["k_static"], x["v_static"], n_static)


def check_decode_dense(seed, n_static=4):
    """K = N and every slot kept: dense attention over all N(1+C) cache rows, the static
    rows and the decode rows (torch SDPA and logsumexp, float64)."""
    B, N, C, Ld, Ls, Hq, Hkv, d = 2, 4, 6, 3, 4, 4, 2, 8
    x = tiny_decode_inputs(seed, B, N, C, Ld, Ls, Hq, Hkv, d)
    ci = np.tile(np.arange(N, dtype=np.int32), (B, 1))
    ts = np.tile(np.arange(1, C + 1, dtype=np.int32), (B, N, 1))
    o, lse = _decode(x, ci, ts, n_static)
    scale = 1.0 / np.sqrt(d)
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            k = np.concatenate([x["k_cache"][b, :, g].reshape(-1, d), x["k_static"][b, :n_static, g], x["k_dec"][b, :, g]])
            v = np.concatenate([x["v_cache"][b, :, g].reshape(-1, d), x["v_static"][b, :n_static, g], x["v_dec"][b, :, g]])
            q = torch.from_numpy(x["q_dec"][b, :, h])
            ot = torch.nn.functional.scaled_dot_product_attention(q[None], torch.from_numpy(k)[None], torch.from_numpy(v)[None])[0]
            np.testing.assert_allclose(o[b, :, h], ot.numpy(), atol=1e-12)
            lt = torch.logsumexp(scale * q @ torch.from_numpy(k).T, dim=1).numpy()
            np.testing.assert_allclose(lse[b, h], lt, atol=1e-12)


def check_decode_permutation(seed):
    """Listing the kept chunks and slots in another order leaves O unchanged."""
    x = tiny_decode_inputs(seed)
    rng = np.random.default_rng(seed)
    ci = np.array([[0, 2], [1, 3]], np.int32)
    ts = np.sort(rng.permuted(np.tile(np.arange(1, 7), (2, 2, 1)), axis=2)[:, :, :3], axis=2).astype(np.int32)
    o1, l1 = _decode(x, ci, ts, 2)
    o2, l2 = _decode(x, ci[:, ::-1].copy(), ts[:, ::-1, ::-1].copy(), 2)
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)


# --- static-selection mode ---------------------------------------------------------------------------------------

def check_static_golden():
    g = _load("static_worked_example.json")
    q_qm = np.array(g["q_qm"], float)
    km = np.array(g["key_mean"], float)
    ts = np.array(g["tok_score"], float)
    dm = g["dims"]
    ci, sl, sc = OT.static_select_ref(q_qm, km, ts, dm["top_k"], dm["tok_budget"], dm["q_len"], dm["scale"])
    np.testing.assert_allclose(sc, np.array(g["expect_scores"], float), atol=1e-12)
    assert np.array_equal(ci, np.array(g["expect_chunk_idx"]))
    assert np.array_equal(sl, np.array(g["expect_tok_slot"]))
    cache = np.zeros((1, 2, 1, 4, 2))
    for n in range(2):
        for slot in range(4):
            cache[0, n, 0, slot] = [10 * n + slot, -(10 * n + slot)]
    np.testing.assert_array_equal(OT.gather_selected_ref(cache, ci, sl), np.array(g["expect_k_sel"], float))


def _tiny_selection(seed, B, N, C, K, Bt):
    rng = np.random.default_rng(seed + 100)
    ci = np.stack([np.sort(rng.permutation(N)[:K]) for _ in range(B)]).astype(np.int32)
    ts = np.stack([np.stack([np.sort(rng.permutation(C)[:Bt] + 1) for _ in range(K)]) for _ in range(B)])
    return ci, ts.astype(np.int32)


def check_gather_matches_decode_rows(seed):
    """The compact rows of (b, g) are the first K(1+B_tok) rows the per-step decode reads."""
    B, N, C, Hkv, d, K, Bt = 2, 4, 6, 2, 8, 2, 3
    x = tiny_decode_inputs(seed, B, N, C, 3, 4, 4, Hkv, d)
    ci, ts = _tiny_selection(seed, B, N, C, K, Bt)
    ks = OT.gather_selected_ref(x["k_cache"], ci, ts)
    for b in range(B):
        for g in range(Hkv):
            rows = OD.decode_kv_rows(x["k_cache"], x["k_static"], x["k_dec"], ci, ts, 0, b, g)
            np.testing.assert_array_equal(ks[b, g], rows[:K * (1 + Bt)])


def check_compact_decode_equals_gathered(seed, n_static):
    """Decode over the compacted rows equals the per-step decode with the same selection."""
    B, N, C, Hkv, d, K, Bt = 2, 4, 6, 2, 8, 3, 4
    x = tiny_decode_inputs(seed, B, N, C, 3, 4, 4, Hkv, d)
    ci, ts = _tiny_selection(seed, B, N, C, K, Bt)
    ks, vs = OT.gather_selected_ref(x["k_cache"], ci, ts), OT.gather_selected_ref(x["v_cache"], ci, ts)
    o1, l1 = OT.decode_compact_ref(x["q_dec"], x["k_dec"], x["v_dec"], ks, vs, x["k_static"], x["v_static"], n_static)
    o2, l2 = _decode(x, ci, ts, n_static)
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)


def check_compact_decode_sdpa(seed):
    """An arbitrary compact buffer: dense attention over [compact ; static ; own] (torch SDPA, float64)."""
    B, Ld, Ls, Hq, Hkv, d, n_sel, n_static = 2, 3, 4, 4, 2, 8, 5, 3
    rng = np.random.default_rng(seed)
    x = tiny_decode_inputs(seed, B, 2, 2, Ld, Ls, Hq, Hkv, d)
    ks, vs = rng.standard_normal((B, Hkv, n_sel, d)), rng.standard_normal((B, Hkv, n_sel, d))
    o, lse = OT.decode_compact_ref(x["q_dec"], x["k_dec"], x["v_dec"], ks, vs, x["k_static"], x["v_static"], n_static)
    scale = 1.0 / np.sqrt(d)
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            k = np.concatenate([ks[b, g], x["k_static"][b, :n_static, g], x["k_dec"][b, :, g]])
            v = np.concatenate([vs[b, g], x["v_static"][b, :n_static, g], x["v_dec"][b, :, g]])
            q = torch.from_numpy(x["q_dec"][b, :, h])
            ot = torch.nn.functional.scaled_dot_product_attention(q[None], torch.from_numpy(k)[None],
                                                                  torch.from_numpy(v)[None])[0]
            np.testing.assert_allclose(o[b, :, h], ot.numpy(), atol=1e-12)
            lt = torch.logsumexp(scale * q @ torch.from_numpy(k).T, dim=1).numpy()
            np.testing.assert_allclose(lse[b, h], lt, atol=1e-12)
