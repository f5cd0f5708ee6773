"""A seeded sweep of random problem shapes through the whole per-step path on the
GPU: prefill (every unit against the oracle), selection from the GPU's own
chunk means (scores against the oracle's, from the inputs; chunk sets by rule
A; token sets exactly those of the GPU token ranks, which the prefill check
holds against the oracle's scores) and decode with the GPU's selection (against the
oracle run on the same indices).  Shapes are drawn from the ranges the C ABI
accepts, small enough for the oracle: dtype, batch, chunk count and length
(ragged), query and pseudo-label lengths, heads per KV head, head dim, K and
B_tok, shared or per-chunk q/m rows, static rows, shard count.  Tolerances as
in test_gpu_parity.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_path import (check_topk_rule_a, h64, random_decode_inputs, random_prefill_inputs, run_decode,
                      run_prefill, run_select)
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims
from test_gpu_parity import decode_check, prefill_units_check

pytestmark = pytest.mark.gpu


def draw(i):
    rng = np.random.default_rng(1000 + i)
    dt = PD_BF16 if rng.random() < 0.75 else PD_FP32
    N = int(rng.integers(1, 7))
    C = int(rng.choice([1, 7, 31, 64, 65, 100, 128, 191, 300]))
    G = int(rng.choice([1, 2, 4, 7]))
    Hkv = int(rng.integers(1, 3))
    Lq = int(rng.integers(1, 41))
    Lm = int(rng.integers(0, 41))
    n_static = int(rng.choice([0, Lq, Lq + Lm]))
    return dict(dt=dt, B=int(rng.integers(1, 3)), N=N, C=C, Lq=Lq, Lm=Lm, Ld=int(rng.integers(1, 71)),
                Hq=G * Hkv, Hkv=Hkv, D=int(rng.choice([64, 128])), K=int(rng.integers(1, N + 1)),
                Bt=int(rng.integers(1, C + 1)), pc=int(rng.integers(0, 2)), n_static=n_static,
                splits=int(rng.choice([0, 1, 3])))


@pytest.mark.parametrize("i", range(48))
def test_random_shape_path(i):
    c = draw(i)
    print(f"[sweep {i}] {c}", flush=True)
    d = Dims(c["B"], c["N"], c["C"], c["Lq"], c["Lm"], c["Ld"], c["Hq"], c["Hkv"], c["D"], c["dt"], 0.0, c["pc"])
    sc = 1.0 if c["dt"] == PD_BF16 else 0.125
    x = random_prefill_inputs(d, seed=2000 + i, scale=sc)
    out = run_prefill(d, x)
    dec = random_decode_inputs(d, seed=3000 + i, scale=sc)
    ci, ts, cs = run_select(d, c["K"], c["Bt"], dec["q_dec"], out["key_mean"], out["tok_rank"])
    torch.cuda.synchronize()
    prefill_units_check(d, x, out, [(b, n) for b in range(d.batch) for n in range(d.n_chunks)])
    s_ref = oracle.chunk_scores_ref(h64(dec["q_dec"]), oracle.key_mean_ref(h64(x["k_pre"])))
    np.testing.assert_allclose(h64(cs), s_ref, rtol=1e-5, atol=1e-5)
    for b in range(d.batch):
        check_topk_rule_a(s_ref[b], ci[b].cpu().numpy(), c["K"])
    want = oracle.tokens_by_rank_ref(out["tok_rank"].cpu().numpy(), ci.cpu().numpy(), c["Bt"])
    assert np.array_equal(ts.cpu().numpy(), want)
    # Static rows in the shared [B][L_q+L_m][H_kv][d] layout (chunk 0's copy when per chunk), contiguous.
    kst = (x["k_qm"][:, 0] if c["pc"] else x["k_qm"]).contiguous()
    vst = (x["v_qm"][:, 0] if c["pc"] else x["v_qm"]).contiguous()
    o, lse = run_decode(d, c["K"], c["Bt"], dec, out, ci, ts, kst, vst, c["n_static"], num_splits=c["splits"])
    torch.cuda.synchronize()
    # The oracle reads the cache as the inputs' rows in cache layout (the GPU cache is checked bit for bit above).
    cache_ref = {n: x[p].permute(0, 1, 3, 2, 4).contiguous() for n, p in (("k_cache", "k_pre"), ("v_cache", "v_pre"))}
    decode_check(d, c["K"], c["Bt"], dec, cache_ref, ci, ts, kst, vst, c["n_static"], o, lse)
