"""GPU parity of the prefill-time chunk score, the query-to-chunk token score and
selection from given chunk scores, against the fp64 oracle, through the C ABI.

Tolerances.  The chunk score is -ln of a head-averaged mass ratio, so its error
is the ratio's relative error: the kernels' logits differ from the fp64 ones by
fp32 accumulation and the exponentials by a few ulp, and the mass and row sums
are fp32 sums of up to S_c positive terms (relative error <= S_c * 2^-24, about
1e-4 at S_c = 1665).  Each of the two terms is a mean of such errors, hence an
absolute bound of 2e-4 for bf16 inputs.  fp32 inputs keep the same sums: 2e-4.
Token scores: 1e-4 absolute, as for the two-sided score.  Selection from given
scores is integer work on identical fp32 inputs: bit-exact.  Selection from
the GPU's own chunk scores: rule A against the oracle's scores (exact wherever
the oracle's gap exceeds 1e-3).
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from gpu_path import check_rank_consistent, check_topk_rule_a, h64, random_prefill_inputs, run_prefill
from paper_2606_10537_amd import _lib, synth
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims
from test_gpu_parity import bits

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
SCORE_ATOL = 2e-4


def run_select_ranked(d, top_k, tok_budget, chunk_score, lowest, tok_rank):
    dev = chunk_score.device
    ci = torch.full((d.batch, top_k), -1, dtype=torch.int32, device=dev)
    ts = torch.full((d.batch, top_k, tok_budget), -1, dtype=torch.int32, device=dev)
    _lib.pd_select_ranked(d, top_k, tok_budget, chunk_score, lowest, tok_rank, ci, ts)
    return ci, ts


def unit_inputs(d, x, b, n):
    return {k: h64(v[b:b + 1, n:n + 1] if (k.endswith("_pre") or d.qm_per_chunk) else v[b:b + 1])
            for k, v in x.items()}


def oracle_unit(d, xs):
    """(content mass (Hq, Lq+Lm), e (C,), e_q2c (C,)) of one (b, n) over all heads."""
    mass = np.zeros((d.n_heads_q, d.q_len + d.m_len))
    e = np.zeros(d.chunk_len)
    e_q2c = np.zeros(d.chunk_len)
    for h in range(d.n_heads_q):
        u = oracle.prefill_unit_ref(xs["q_pre"], xs["k_pre"], xs["v_pre"], xs["q_qm"], xs["k_qm"], xs["v_qm"],
                                    0, 0, h, d.q_len, d.sm_scale)
        mass[h] = u["content_mass"]
        e += u["e_head"]
        e_q2c += u["e_q2c_head"]
    return mass, e, e_q2c


CASES = [
    # dtype, B, N, C, Lq, Lm, Hq, Hkv, D, per_chunk
    (PD_BF16, 2, 3, 128, 16, 32, 4, 4, 64, 0),
    (PD_BF16, 1, 2, 300, 40, 0, 4, 2, 128, 0),       # L_m = 0: the query term only; ragged tiles
    (PD_BF16, 1, 2, 1000, 64, 200, 2, 1, 128, 1),    # several row tiles; q rows start inside a wave
    (PD_BF16, 1, 1, 1, 1, 1, 1, 1, 128, 0),          # smallest chunk
    (PD_FP32, 1, 3, 77, 9, 3, 4, 2, 128, 1),
    (PD_FP32, 2, 2, 64, 16, 16, 2, 2, 64, 0),
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_chunk_score_parity(case):
    """Chunk score of every (b, n) against the oracle; every other output bit-identical
    to a call without the chunk score."""
    dt, B, N, C, Lq, Lm, Hq, Hkv, D, pc = case
    d = Dims(B, N, C, Lq, Lm, 8, Hq, Hkv, D, dt, 0.0, pc)
    print(f"[chunk score] {case}", flush=True)
    x = random_prefill_inputs(d, seed=hash(case) % 10000, scale=1.0 if dt == PD_BF16 else 0.25)
    out = run_prefill(d, x, chunk_score=True)
    ref = run_prefill(d, x)
    torch.cuda.synchronize()
    for k in ref:
        assert np.array_equal(bits(out[k]), bits(ref[k])), k
    s_ref = np.zeros((B, N))
    for b in range(B):
        for n in range(N):
            mass, _, _ = oracle_unit(d, unit_inputs(d, x, b, n))
            s_ref[b, n] = oracle.prefill_chunk_score_ref(mass[None, None], Lq)[0, 0]
    np.testing.assert_allclose(h64(out["chunk_score"]), s_ref, rtol=0, atol=SCORE_ATOL)


@pytest.mark.parametrize("case", [CASES[0], CASES[2], CASES[4], (PD_BF16, 1, 2, 96, 200, 10, 4, 2, 128, 0)],
                         ids=["bf16-small", "bf16-tiles", "fp32", "bf16-200-query-rows"])
def test_query_to_chunk_token_score(case):
    dt, B, N, C, Lq, Lm, Hq, Hkv, D, pc = case
    d = Dims(B, N, C, Lq, Lm, 8, Hq, Hkv, D, dt, 0.0, pc, tok_score_dir=1)
    x = random_prefill_inputs(d, seed=77, scale=1.0 if dt == PD_BF16 else 0.25)
    out = run_prefill(d, x)
    torch.cuda.synchronize()
    for b in range(B):
        for n in range(N):
            _, _, e_q2c = oracle_unit(d, unit_inputs(d, x, b, n))
            np.testing.assert_allclose(h64(out["tok_score"][b, n]), e_q2c, rtol=0, atol=1e-4)
            check_rank_consistent(e_q2c, out["tok_rank"][b, n].cpu().numpy())


def test_chunk_score_golden_fp32():
    """The hand-derived two-head example, zero-padded from d = 2 to d = 64."""
    g = json.load(open(os.path.join(GOLDEN, "chunk_score_worked_example.json")))
    x = {}
    for k in ("q_pre", "k_pre", "v_pre", "q_qm", "k_qm", "v_qm"):
        a = np.array(g[k], dtype=np.float32)
        pad = np.zeros(a.shape[:-1] + (64,), np.float32)
        pad[..., :2] = a
        x[k] = torch.from_numpy(pad).cuda()
    for direction, key in ((0, "expect_tok_score"), (1, "expect_tok_score_q2c")):
        d = Dims(1, 1, 1, 1, 1, 1, 2, 2, 64, PD_FP32, 1.0, 0, tok_score_dir=direction)
        out = run_prefill(d, x, chunk_score=True)
        torch.cuda.synchronize()
        assert abs(h64(out["chunk_score"])[0, 0] - np.log(float(Fraction(g["expect_chunk_score_exp"])))) < 1e-6
        np.testing.assert_allclose(h64(out["tok_score"][0, 0]), [float(Fraction(v)) for v in g[key]], atol=1e-6)


def test_select_ranked_golden():
    g = json.load(open(os.path.join(GOLDEN, "chunk_score_worked_example.json")))["select"]
    cs = torch.tensor(g["chunk_score"], dtype=torch.float32, device="cuda")
    tr = torch.tensor(g["tok_rank"], dtype=torch.int32, device="cuda")
    d = Dims(1, 4, 3, 1, 1, 1, 1, 1, 64, PD_FP32)
    for case in g["cases"]:
        ci, ts = run_select_ranked(d, case["top_k"], g["tok_budget"], cs, case["lowest"], tr)
        assert ci.cpu().tolist() == case["chunk_idx"], case
        assert ts.cpu().tolist() == case["tok_slot"], case


@pytest.mark.parametrize("B,N,C,K,Bt", [(2, 7, 33, 3, 5), (3, 1024, 16, 4, 16), (1, 1024, 1024, 1024, 1),
                                         (2, 5, 4096, 5, 4096), (1, 1, 1, 1, 1)])
def test_select_ranked_parity(B, N, C, K, Bt):
    """Identical fp32 scores with many ties (and +-0): bit-exact chunk and slot lists."""
    rng = np.random.default_rng(B * 1000 + N + C)
    cs = rng.integers(-3, 4, size=(B, N)).astype(np.float32) * 0.5
    cs[cs == 0] = np.where(rng.random(np.count_nonzero(cs == 0)) < 0.5, -0.0, 0.0)
    tr = np.stack([np.stack([rng.permutation(C) for _ in range(N)]) for _ in range(B)]).astype(np.int32)
    d = Dims(B, N, C, 1, 1, 1, 1, 1, 64, PD_BF16)
    cs_d = torch.from_numpy(cs).cuda()
    tr_d = torch.from_numpy(tr).cuda()
    for lowest in (1, 0):
        ci, ts = run_select_ranked(d, K, Bt, cs_d, lowest, tr_d)
        ci_ref, ts_ref = oracle.select_ranked_ref(cs, tr, K, Bt, lowest=bool(lowest))
        assert np.array_equal(ci.cpu().numpy(), ci_ref)
        assert np.array_equal(ts.cpu().numpy(), ts_ref)


def test_prefill_score_then_select_end_to_end():
    """Chunk scores from the prefill, the K lowest kept: rule A against the oracle's
    scores, kept slots exactly those the GPU's own token ranks give."""
    d = Dims(2, 6, 200, 24, 40, 8, 4, 2, 128, PD_BF16)
    x = random_prefill_inputs(d, seed=31)
    out = run_prefill(d, x, chunk_score=True)
    ci, ts = run_select_ranked(d, 3, 50, out["chunk_score"], 1, out["tok_rank"])
    torch.cuda.synchronize()
    for b in range(d.batch):
        s_ref = np.array([oracle.prefill_chunk_score_ref(oracle_unit(d, unit_inputs(d, x, b, n))[0][None, None],
                                                         d.q_len)[0, 0] for n in range(d.n_chunks)])
        check_topk_rule_a(-s_ref, ci[b].cpu().numpy(), 3)
    assert np.array_equal(ts.cpu().numpy(),
                          oracle.tokens_by_rank_ref(out["tok_rank"].cpu().numpy(), ci.cpu().numpy(), 50))


@pytest.mark.parametrize("wid,units", [(2, [(0, 0), (0, 5)]), (5, [(0, 0), (7, 31)])])
def test_workload_chunk_score_sampled(wid, units):
    """Full-size layer in the launch configuration bench.py times: sampled (b, n)
    chunk scores against the oracle over every head, the K lowest by rule A where
    the whole row of scores is known, and (planted workload) the planted chunks kept."""
    w = synth.WORKLOADS[wid]
    d = w.dims()
    x = synth.make_prefill(w, 0, "cuda")
    out = run_prefill(d, x, chunk_score=True)
    ci, _ = run_select_ranked(d, w.top_k, w.tok_budget, out["chunk_score"], 1, out["tok_rank"])
    torch.cuda.synchronize()
    got = h64(out["chunk_score"])
    assert np.all(np.isfinite(got))
    for (b, n) in units:
        print(f"[workload {wid}] chunk score unit {(b, n)}", flush=True)
        mass, _, _ = oracle_unit(d, unit_inputs(d, x, b, n))
        s_ref = oracle.prefill_chunk_score_ref(mass[None, None], d.q_len)[0, 0]
        assert abs(got[b, n] - s_ref) <= SCORE_ATOL, (b, n, got[b, n], s_ref)
    # The selection is exactly the K lowest of the GPU's own scores (ties to the lower index).
    ci_own, _ = oracle.select_ranked_ref(got, out["tok_rank"].cpu().numpy(), w.top_k, w.tok_budget)
    assert np.array_equal(ci.cpu().numpy(), ci_own)
    pl = synth.plant_info(w, 0)
    if pl is not None:
        for b in range(d.batch):
            assert set(pl["chunks"][b]) <= set(ci[b].cpu().tolist())
