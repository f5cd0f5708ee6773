"""GPU parity: every C-ABI entry point against the fp64 oracle on the same inputs.

Tolerances (from the method's acceptance rules): outputs max-abs <= 1e-2 for
bf16 inputs and <= 1e-5 for fp32 inputs; the chunk cache bit-exact; key means
within relative 1e-5; token scores within 1e-4 absolute; chunk and token index
sets by rule A (exact wherever the oracle's score gap exceeds 1e-3); decode
outputs checked with the oracle run on the GPU's own indices.
"""

import json
import os

import numpy as np
import pytest
import torch

import oracle
from gpu_path import (check_rank_consistent, check_topk_rule_a, h64, random_decode_inputs, random_indices,
                      random_prefill_inputs, run_decode, run_prefill, run_select)
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TOL = {PD_BF16: 1e-2, PD_FP32: 1e-5}


def assert_out_close(d, got, ref, what):
    """max-abs <= 1e-2 (bf16 inputs) or 1e-5 (fp32 inputs); when the output itself is
    stored as bf16, each element may also carry its rounding, <= 2^-8 |O|."""
    err = np.abs(got - ref)
    bound = TOL[d.dtype] + (2.0 ** -8 * np.abs(ref) if d.dtype == PD_BF16 and not d.out_fp32 else 0.0)
    worst = np.max(err - bound)
    assert worst <= 0, f"{what}: max-abs {err.max():.3g} exceeds the bound by {worst:.3g}"


def assert_lse_close(d, got, ref, q, k, what):
    """Natural-log row LSE of one (sequence, head): got, ref (L,); q (L, d) the query rows and
    k (M, d) the key rows (or a superset of them) the rows attend to, fp64.

    fp32 inputs: 1e-4 absolute.  bf16 inputs: the weights entering the row sum are
    rounded to bf16 (each within 2^-8 relative: 8 significant bits), so the log of
    the sum is within log(1 + 2^-8); every logit also carries its fp32 accumulation
    error, at most d 2^-23 scale sum_i |q_i k_i| (d products, doubled for the
    matrix cores' accumulation order), which shifts the LSE by at most its
    largest value over the row's keys.  The bound per row is the sum of the two."""
    if d.dtype == PD_BF16:
        scale = d.sm_scale if d.sm_scale > 0 else 1.0 / np.sqrt(d.head_dim)
        logit_err = d.head_dim * 2.0 ** -23 * scale * (np.abs(q) @ np.abs(k).T).max(axis=1)
        bound = np.log1p(2.0 ** -8) + logit_err + 1e-6
    else:
        bound = 1e-4
    err = np.abs(np.asarray(got) - ref)
    worst = np.max(err - bound)
    assert worst <= 0, f"{what}: LSE error {err.max():.3g} exceeds the bound by {worst:.3g}"


def bits(t):
    """Raw element bits of a host tensor (bf16 -> int16, fp32 -> int32)."""
    t = t.detach().cpu()
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).numpy()


def prefill_units_check(d, x, out, units, check_e=True):
    """Oracle check of the listed (b, n) units: O for every head, cache bits, key mean, e."""
    for (b, n) in units:
        xs = {k: h64(v[b:b + 1, n:n + 1] if (k.endswith("_pre") or d.qm_per_chunk) else v[b:b + 1])
              for k, v in x.items()}
        e = np.zeros(d.chunk_len)
        for h in range(d.n_heads_q):
            u = oracle.prefill_unit_ref(xs["q_pre"], xs["k_pre"], xs["v_pre"], xs["q_qm"], xs["k_qm"], xs["v_qm"],
                                        0, 0, h, d.q_len, d.sm_scale)
            assert_out_close(d, h64(out["o"][b, n, :, h]), u["o"], f"prefill O (b={b}, n={n}, h={h})")
            e += u["e_head"]
        assert np.array_equal(bits(out["k_cache"][b, n]), oracle.cache_ref(bits(x["k_pre"][b:b + 1, n:n + 1]))[0, 0])
        assert np.array_equal(bits(out["v_cache"][b, n]), oracle.cache_ref(bits(x["v_pre"][b:b + 1, n:n + 1]))[0, 0])
        km = oracle.key_mean_ref(xs["k_pre"])[0, 0]
        np.testing.assert_allclose(h64(out["key_mean"][b, n]), km, rtol=1e-5, atol=1e-6 * np.abs(km).max())
        if check_e:
            np.testing.assert_allclose(h64(out["tok_score"][b, n]), e, rtol=0, atol=1e-4)
            check_rank_consistent(e, out["tok_rank"][b, n].cpu().numpy())


# --------------------------------------------------------------------------- stage (a)

PREFILL_CASES = [
    # dtype, B, N, C, Lq, Lm, Hq, Hkv, D, per_chunk
    (PD_BF16, 2, 3, 128, 16, 32, 4, 4, 64, 0),
    (PD_BF16, 1, 2, 100, 17, 5, 4, 2, 128, 0),
    (PD_BF16, 2, 2, 200, 40, 0, 6, 1, 128, 1),
    (PD_BF16, 1, 3, 64, 64, 63, 2, 2, 64, 0),
    (PD_BF16, 1, 1, 1, 1, 0, 1, 1, 128, 0),
    (PD_BF16, 1, 2, 96, 200, 10, 7, 1, 128, 0),        # L_q > 128: several query-row passes; 7 heads per KV head
    (PD_BF16, 1, 2, 33, 300, 0, 4, 4, 64, 1),          # L_q > 256, d = 64, per-chunk q/m rows
    (PD_BF16 + 10, 1, 2, 130, 20, 9, 4, 2, 128, 0),     # bf16 inputs, fp32 outputs
    (PD_FP32, 1, 4, 128, 16, 32, 4, 4, 64, 0),
    (PD_FP32, 2, 2, 77, 9, 3, 4, 2, 128, 1),
    (PD_FP32, 1, 1, 1, 1, 0, 1, 1, 64, 0),
]


@pytest.mark.parametrize("case", PREFILL_CASES, ids=[str(c) for c in PREFILL_CASES])
def test_prefill_parity(case):
    dt, B, N, C, Lq, Lm, Hq, Hkv, D, pc = case
    d = Dims(B, N, C, Lq, Lm, 8, Hq, Hkv, D, dt % 10, 0.0, pc, out_fp32=int(dt >= 10))
    dt = dt % 10
    x = random_prefill_inputs(d, seed=hash(case) % 10000, scale=1.0 if dt == PD_BF16 else 0.125)
    out = run_prefill(d, x)
    torch.cuda.synchronize()
    prefill_units_check(d, x, out, [(b, n) for b in range(B) for n in range(N)])


def test_prefill_golden_fp32():
    """The hand-derived worked example, zero-padded from d = 2 to d = 64 (dot products unchanged)."""
    g = json.load(open(os.path.join(GOLDEN, "prefill_worked_example.json")))
    d = Dims(1, 1, 2, 1, 1, 1, 1, 1, 64, PD_FP32, 1.0, 0)
    x = {}
    for k in ("q_pre", "k_pre", "v_pre", "q_qm", "k_qm", "v_qm"):
        a = np.array(g[k], dtype=np.float32)
        pad = np.zeros(a.shape[:-1] + (64,), np.float32)
        pad[..., :2] = a
        x[k] = torch.from_numpy(pad).cuda()
    out = run_prefill(d, x)
    torch.cuda.synchronize()
    from fractions import Fraction
    want = np.array([[float(Fraction(v)) for v in row] for row in g["expect_o_rows"]])
    np.testing.assert_allclose(h64(out["o"][0, 0, :, 0, :2]), want, atol=1e-6)
    assert np.all(h64(out["o"][0, 0, :, 0, 2:]) == 0)
    np.testing.assert_allclose(h64(out["tok_score"][0, 0]), [float(Fraction(v)) for v in g["expect_tok_score"]],
                               atol=1e-6)
    np.testing.assert_allclose(h64(out["key_mean"][0, 0, 0, :2]), g["expect_key_mean"], atol=1e-7)


def test_prefill_deterministic():
    d = Dims(1, 3, 300, 20, 10, 8, 4, 2, 128, PD_BF16)
    x = random_prefill_inputs(d, seed=5)
    a = run_prefill(d, x)
    b = run_prefill(d, x)
    torch.cuda.synchronize()
    for k in a:
        assert np.array_equal(bits(a[k]), bits(b[k])), k


# --------------------------------------------------------------------------- stage (b)

def test_select_golden():
    g = json.load(open(os.path.join(GOLDEN, "select_worked_example.json")))
    q = np.zeros((1, 2, 2, 64), np.float32)
    q[..., :2] = np.array(g["q_dec"], np.float32)
    km = np.zeros((1, 3, 1, 64), np.float32)
    km[..., :2] = np.array(g["key_mean"], np.float32)
    ts = torch.tensor(g["expect_tok_rank"], dtype=torch.int32).cuda()
    for case in g["cases"]:
        d = Dims(1, 3, 4, 1, 0, 2, 2, 1, 64, PD_FP32, 1.0, 0)
        ci, tsl, cs = run_select(d, case["top_k"], case["tok_budget"], torch.from_numpy(q).cuda(),
                                 torch.from_numpy(km).cuda(), ts)
        torch.cuda.synchronize()
        assert ci.cpu().tolist() == [case["chunk_idx"]]
        assert tsl.cpu().tolist() == [case["tok_slot"]]
        np.testing.assert_allclose(h64(cs)[0], g["expect_scores"], atol=1e-6)


SELECT_CASES = [
    # dtype, B, N, C, Ld, Hq, Hkv, D, K, Bt
    (PD_BF16, 2, 8, 1024, 64, 8, 8, 128, 2, 512),
    (PD_BF16, 1, 16, 1024, 32, 7, 1, 128, 4, 256),
    (PD_BF16, 3, 5, 100, 17, 4, 2, 64, 5, 100),     # K = N, Bt = C
    (PD_BF16, 1, 1, 33, 3, 2, 2, 64, 1, 1),
    (PD_FP32, 2, 40, 300, 9, 4, 4, 64, 7, 33),
    (PD_FP32, 1, 1024, 16, 4, 2, 1, 64, 10, 16),
    (PD_BF16, 2, 100, 40, 20, 4, 2, 64, 80, 9),     # K > 64: the two-launch selection
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=[str(c) for c in SELECT_CASES])
def test_select_parity(case):
    dt, B, N, C, Ld, Hq, Hkv, D, K, Bt = case
    d = Dims(B, N, C, 4, 0, Ld, Hq, Hkv, D, dt)
    g = torch.Generator().manual_seed(hash(case) % 10000)
    tdt = torch.bfloat16 if dt == PD_BF16 else torch.float32
    q = (torch.randn((B, Ld, Hq, D), generator=g) + 0.3 * torch.randn((1, 1, Hq, D), generator=g)).to(tdt).cuda()
    km = torch.randn((B, N, Hkv, D), generator=g).cuda()
    rank = torch.argsort(torch.rand((B, N, C), generator=g), dim=2).to(torch.int32).cuda()
    ci, tsl, cs = run_select(d, K, Bt, q, km, rank)
    torch.cuda.synchronize()
    s_ref = oracle.chunk_scores_ref(h64(q), h64(km))
    np.testing.assert_allclose(h64(cs), s_ref, rtol=1e-5, atol=1e-5)
    for b in range(B):
        check_topk_rule_a(s_ref[b], ci[b].cpu().numpy(), K)
    want = oracle.tokens_by_rank_ref(rank.cpu().numpy(), ci.cpu().numpy(), Bt)
    assert np.array_equal(tsl.cpu().numpy(), want)


def test_select_repeated_calls_one_workspace():
    """Calls in a row on one workspace (different batch sizes and K) each match the oracle: nothing a call
    leaves in the workspace leaks into the next."""
    from gpu_path import workspace
    from paper_2606_10537_amd import _lib
    g = torch.Generator().manual_seed(77)
    big = Dims(6, 12, 64, 4, 0, 300, 8, 4, 64, PD_BF16)
    ws = workspace(_lib.pd_workspace_bytes(big, 12, 64, 0, 1))
    for it, (B, K) in enumerate([(6, 3), (2, 5), (6, 12), (4, 1), (6, 3)]):
        d = Dims(B, 12, 64, 4, 0, 300, 8, 4, 64, PD_BF16)
        q = torch.randn((B, 300, 8, 64), generator=g).to(torch.bfloat16).cuda()
        km = torch.randn((B, 12, 4, 64), generator=g).cuda()
        rank = torch.argsort(torch.rand((B, 12, 64), generator=g), dim=2).to(torch.int32).cuda()
        ci = torch.full((B, K), -1, dtype=torch.int32, device="cuda")
        ts = torch.full((B, K, 20), -1, dtype=torch.int32, device="cuda")
        cs = torch.full((B, 12), float("nan"), dtype=torch.float32, device="cuda")
        _lib.pd_score_select(d, K, 20, q, km, rank, ci, ts, cs, ws)
        torch.cuda.synchronize()
        s_ref = oracle.chunk_scores_ref(h64(q), h64(km))
        np.testing.assert_allclose(h64(cs), s_ref, rtol=1e-5, atol=1e-5)
        for b in range(B):
            check_topk_rule_a(s_ref[b], ci[b].cpu().numpy(), K)
        assert np.array_equal(ts.cpu().numpy(), oracle.tokens_by_rank_ref(rank.cpu().numpy(), ci.cpu().numpy(), 20))


def test_prefill_then_select_end_to_end():
    """Token selection through the prefill's ranks agrees with the oracle's top-B by Eq. 5 (rule A)."""
    d = Dims(2, 5, 300, 24, 8, 16, 4, 2, 128, PD_BF16)
    x = random_prefill_inputs(d, seed=31)
    out = run_prefill(d, x)
    q = random_decode_inputs(d, seed=32)["q_dec"]
    ci, tsl, cs = run_select(d, 3, 100, q, out["key_mean"], out["tok_rank"])
    torch.cuda.synchronize()
    xs = {k: h64(v) for k, v in x.items()}
    ref = oracle.prefill_ref(xs["q_pre"], xs["k_pre"], xs["v_pre"], xs["q_qm"], xs["k_qm"], xs["v_qm"], d.q_len)
    s_ref = oracle.chunk_scores_ref(h64(q), ref["key_mean"])
    for b in range(2):
        check_topk_rule_a(s_ref[b], ci[b].cpu().numpy(), 3)
        for kk, n in enumerate(ci[b].cpu().tolist()):
            check_topk_rule_a(ref["tok_score"][b, n], tsl[b, kk].cpu().numpy() - 1, 100)


def test_select_ties_and_zero_query():
    """Q_dec = 0 gives all-zero scores: the first K chunks; identity ranks: the first Bt slots."""
    d = Dims(2, 9, 50, 4, 0, 8, 4, 2, 64, PD_BF16)
    q = torch.zeros((2, 8, 4, 64), dtype=torch.bfloat16).cuda()
    km = torch.randn((2, 9, 2, 64)).cuda()
    rank = torch.arange(50, dtype=torch.int32).cuda().repeat(2, 9, 1)
    ci, tsl, cs = run_select(d, 3, 7, q, km, rank)
    torch.cuda.synchronize()
    assert ci.cpu().tolist() == [[0, 1, 2]] * 2
    assert tsl.cpu().tolist() == [[list(range(1, 8))] * 3] * 2


# --------------------------------------------------------------------------- stage (c)

def decode_check(d, K, Bt, dec, cache, ci, ts, k_static, v_static, n_static, o, lse, heads=None, batches=None):
    cih, tsh = ci.cpu().numpy(), ts.cpu().numpy()
    for b in (batches if batches is not None else range(d.batch)):
        # Only the selected chunks of sequence b reach the oracle (same rows, re-indexed).
        sel = cih[b].tolist()
        kc = h64(cache["k_cache"][b:b + 1, sel])
        vc = h64(cache["v_cache"][b:b + 1, sel])
        ks = h64(k_static[b:b + 1]) if n_static else np.zeros((1, 0, d.n_heads_kv, d.head_dim))
        vs = h64(v_static[b:b + 1]) if n_static else np.zeros((1, 0, d.n_heads_kv, d.head_dim))
        dq, dk, dv = (h64(dec[n][b:b + 1]) for n in ("q_dec", "k_dec", "v_dec"))
        ci0 = np.arange(K, dtype=np.int32)[None]
        for h in (heads if heads is not None else range(d.n_heads_q)):
            ro, rl = oracle.decode_unit_ref(dq, dk, dv, kc, vc, ci0, tsh[b:b + 1], ks, vs, n_static, 0, h,
                                            d.sm_scale)
            assert_out_close(d, h64(o[b, :, h]), ro, f"decode O (b={b}, h={h})")
            if lse is not None:
                # Keys: every row of the kept chunks (a superset of the kept rows),
                # the static rows and the own rows.
                g = h // (d.n_heads_q // d.n_heads_kv)
                keys = np.concatenate([kc[0, :, g].reshape(-1, d.head_dim), ks[0, :n_static, g], dk[0, :, g]])
                assert_lse_close(d, h64(lse[b, h]), rl, dq[0, :, h], keys, f"decode LSE (b={b}, h={h})")


DECODE_CASES = [
    # dtype, B, N, C, Lq, Lm, Ld, Hq, Hkv, D, K, Bt, n_static, splits
    (PD_BF16, 2, 4, 128, 16, 32, 32, 4, 4, 64, 2, 100, 16, 1),
    (PD_BF16, 1, 6, 200, 20, 0, 70, 4, 2, 128, 3, 150, 20, 3),
    (PD_BF16, 2, 5, 64, 8, 8, 1, 7, 1, 128, 5, 64, 0, 0),
    (PD_BF16, 1, 3, 300, 30, 2, 130, 8, 8, 128, 2, 77, 32, 0),
    (PD_BF16, 1, 3, 300, 30, 2, 130, 8, 8, 128, 2, 77, 32, 7),
    (PD_BF16 + 10, 1, 3, 300, 30, 2, 130, 8, 8, 128, 2, 77, 32, 1),   # fp32 outputs
    (PD_BF16 + 10, 1, 3, 300, 30, 2, 130, 8, 8, 128, 2, 77, 32, 3),
    (PD_FP32, 1, 4, 128, 16, 32, 32, 4, 4, 64, 2, 128, 16, 1),
    (PD_FP32, 2, 3, 90, 5, 5, 40, 4, 2, 128, 2, 30, 10, 4),
    (PD_FP32, 1, 2, 16, 4, 0, 1, 2, 1, 64, 1, 1, 0, 0),
]


@pytest.mark.parametrize("case", DECODE_CASES, ids=[str(c) for c in DECODE_CASES])
def test_decode_parity(case):
    dt, B, N, C, Lq, Lm, Ld, Hq, Hkv, D, K, Bt, ns, S = case
    d = Dims(B, N, C, Lq, Lm, Ld, Hq, Hkv, D, dt % 10, out_fp32=int(dt >= 10))
    dt = dt % 10
    sc = 1.0 if dt == PD_BF16 else 0.125
    x = random_prefill_inputs(d, seed=hash(case) % 1000, scale=sc)
    cache = run_prefill(d, x)
    dec = random_decode_inputs(d, seed=hash(case) % 1000 + 1, scale=sc)
    ci, ts = random_indices(d, K, Bt, seed=3)
    o, lse = run_decode(d, K, Bt, dec, cache, ci, ts, x["k_qm"], x["v_qm"], ns, num_splits=S)
    torch.cuda.synchronize()
    decode_check(d, K, Bt, dec, cache, ci, ts, x["k_qm"], x["v_qm"], ns, o, lse)


@pytest.mark.parametrize("dt", [PD_BF16, PD_FP32])
def test_decode_dense_equivalence(dt):
    """K = N and every slot kept: the sparse decode equals dense attention over all prefix rows."""
    d = Dims(1, 3, 64, 8, 8, 16, 4, 2, 64, dt)
    sc = 1.0 if dt == PD_BF16 else 0.125
    x = random_prefill_inputs(d, seed=11, scale=sc)
    cache = run_prefill(d, x)
    dec = random_decode_inputs(d, seed=12, scale=sc)
    ci = torch.arange(3, dtype=torch.int32).cuda()[None]
    ts = torch.arange(1, 65, dtype=torch.int32).cuda().repeat(1, 3, 1)
    o, _ = run_decode(d, 3, 64, dec, cache, ci, ts, x["k_qm"], x["v_qm"], 8)
    torch.cuda.synchronize()
    scale = 1 / np.sqrt(64)
    for h in range(4):
        g = h // 2
        k = np.concatenate([h64(cache["k_cache"][0, :, g]).reshape(-1, 64), h64(x["k_qm"][0, :8, g]), h64(dec["k_dec"][0, :, g])])
        v = np.concatenate([h64(cache["v_cache"][0, :, g]).reshape(-1, 64), h64(x["v_qm"][0, :8, g]), h64(dec["v_dec"][0, :, g])])
        q = h64(dec["q_dec"][0, :, h])
        s = scale * q @ k.T
        p = np.exp(s - s.max(1, keepdims=True))
        ref = (p / p.sum(1, keepdims=True)) @ v
        assert np.abs(h64(o[0, :, h]) - ref).max() <= TOL[dt]


def test_decode_split_invariance():
    """Any shard count gives the same output within rounding (LSE merge of the shards)."""
    d = Dims(1, 4, 256, 16, 0, 64, 4, 4, 128, PD_BF16)
    x = random_prefill_inputs(d, seed=21)
    cache = run_prefill(d, x)
    dec = random_decode_inputs(d, seed=22)
    ci, ts = random_indices(d, 4, 200, seed=23)
    outs = [run_decode(d, 4, 200, dec, cache, ci, ts, x["k_qm"], x["v_qm"], 16, num_splits=s)[0] for s in (1, 2, 5, 13)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert (o.float() - outs[0].float()).abs().max().item() <= 1e-2
