"""GPU parity of the static-selection mode: selection once from the pseudo-label
rows (pd_score_select_static), the kept rows compacted once
(pd_gather_selected), and decode over the compact buffer
(pd_sparse_decode_attn_compact), against the oracle's static module.

* chunk scores relative 1e-4; chunk sets by rule A; token sets exactly those of
  the GPU token ranks (as in the per-step tests);
* the compact buffers bit-exact (a copy);
* the compact decode bit-identical to the per-step decode with the same
  selection (both read the same rows in the same order), and within the
  output tolerance of the oracle for an arbitrary compact buffer, including
  n_sel = 0, a ragged n_sel and Split-S.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_path import (check_topk_rule_a, h64, random_decode_inputs, random_prefill_inputs, run_decode,
                      run_prefill, workspace)
from paper_2606_10537_amd import _lib, synth
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims
from test_gpu_parity import assert_lse_close, assert_out_close, bits

pytestmark = pytest.mark.gpu


def run_static_select(d, K, Bt, q_qm, key_mean, tok_rank):
    ci = torch.full((d.batch, K), -1, dtype=torch.int32, device="cuda")
    ts = torch.full((d.batch, K, Bt), -1, dtype=torch.int32, device="cuda")
    cs = torch.full((d.batch, d.n_chunks), float("nan"), dtype=torch.float32, device="cuda")
    ws = workspace(_lib.pd_workspace_bytes(d, K, Bt, 0, 1))
    _lib.pd_score_select_static(d, K, Bt, q_qm, key_mean, tok_rank, ci, ts, cs, ws)
    return ci, ts, cs


def run_gather(d, K, Bt, cache, ci, ts):
    n_sel = K * (1 + Bt)
    shape = (d.batch, d.n_heads_kv, n_sel, d.head_dim)
    dt = cache["k_cache"].dtype
    ks = torch.full(shape, float("nan"), dtype=dt, device="cuda")
    vs = torch.full(shape, float("nan"), dtype=dt, device="cuda")
    _lib.pd_gather_selected(d, K, Bt, cache["k_cache"], cache["v_cache"], ci, ts, ks, vs)
    return ks, vs


def run_compact(d, n_sel, dec, ks, vs, k_static, v_static, n_static, num_splits=0):
    odt = torch.float32 if d.out_fp32 else dec["q_dec"].dtype
    o = torch.full(dec["q_dec"].shape, float("nan"), dtype=odt, device="cuda")
    lse = torch.full((d.batch, d.n_heads_q, d.dec_len), float("nan"), dtype=torch.float32, device="cuda")
    ws = workspace(_lib.pd_compact_workspace_bytes(d, n_sel, num_splits))
    _lib.pd_sparse_decode_attn_compact(d, n_sel, dec["q_dec"], dec["k_dec"], dec["v_dec"], ks, vs, k_static,
                                       v_static, n_static, o, lse, num_splits, ws)
    return o, lse


STATIC_CASES = [
    # workload, per-chunk q/m rows
    (1, False), (2, False), (3, False), (2, True),
]


@pytest.mark.parametrize("wid,per_chunk", STATIC_CASES)
def test_static_select_gather_compact(wid, per_chunk):
    w = synth.WORKLOADS[wid]
    d = w.dims()
    K, Bt = w.top_k, w.tok_budget
    if per_chunk:
        d.qm_per_chunk = 1
        x = random_prefill_inputs(d, seed=wid + 40, scale=1.0 if d.dtype == PD_BF16 else 0.125)
    else:
        x = synth.make_prefill(w, 0, "cuda")
    out = run_prefill(d, x)
    ci, ts, cs = run_static_select(d, K, Bt, x["q_qm"], out["key_mean"], out["tok_rank"])
    torch.cuda.synchronize()
    print(f"[static {wid} per_chunk={per_chunk}] selection done", flush=True)

    km = h64(out["key_mean"])
    s_ref = oracle.chunk_scores_ref(oracle.pseudo_label_queries(h64(x["q_qm"]), d.q_len), km, d.sm_scale)
    np.testing.assert_allclose(h64(cs), s_ref, rtol=1e-4, atol=1e-4)
    for b in range(d.batch):
        check_topk_rule_a(s_ref[b], ci[b].cpu().numpy(), K)
    assert np.array_equal(ts.cpu().numpy(),
                          oracle.tokens_by_rank_ref(out["tok_rank"].cpu().numpy(), ci.cpu().numpy(), Bt))

    ks, vs = run_gather(d, K, Bt, out, ci, ts)
    torch.cuda.synchronize()
    # A copy: the oracle gathers the raw element bits.
    ref_k = oracle.gather_selected_ref(bits(out["k_cache"]), ci.cpu().numpy(), ts.cpu().numpy())
    ref_v = oracle.gather_selected_ref(bits(out["v_cache"]), ci.cpu().numpy(), ts.cpu().numpy())
    assert np.array_equal(bits(ks), ref_k)
    assert np.array_equal(bits(vs), ref_v)

    dec = synth.make_decode(w, 0, 1, "cuda")
    o1, l1 = run_compact(d, K * (1 + Bt), dec, ks, vs, x["k_qm"], x["v_qm"], w.q_len)
    o2, l2 = run_decode(d, K, Bt, dec, out, ci, ts, x["k_qm"], x["v_qm"], w.q_len)
    torch.cuda.synchronize()
    assert np.array_equal(bits(o1), bits(o2)), "compact decode differs from the gathered decode"
    assert np.array_equal(bits(l1), bits(l2))


COMPACT_CASES = [
    # dtype, B, Ld, Hq, Hkv, D, n_sel, Lq, n_static, splits
    (PD_BF16, 2, 40, 4, 2, 128, 77, 16, 16, 1),
    (PD_BF16, 1, 130, 8, 8, 128, 0, 16, 16, 0),
    (PD_BF16, 1, 33, 4, 4, 64, 300, 8, 0, 3),
    (PD_BF16 + 10, 1, 70, 4, 1, 128, 129, 8, 8, 2),   # fp32 outputs
    (PD_FP32, 2, 40, 4, 2, 64, 77, 16, 16, 1),
    (PD_FP32, 1, 33, 4, 4, 128, 0, 8, 8, 3),
]


@pytest.mark.parametrize("case", COMPACT_CASES, ids=[str(c) for c in COMPACT_CASES])
def test_compact_decode_parity(case):
    dt, B, Ld, Hq, Hkv, D, n_sel, Lq, n_static, splits = case
    d = Dims(batch=B, n_chunks=1, chunk_len=8, q_len=Lq, m_len=4, dec_len=Ld, n_heads_q=Hq, n_heads_kv=Hkv,
             head_dim=D, dtype=dt % 10, out_fp32=1 if dt >= 10 else 0)
    tdt = torch.bfloat16 if d.dtype == PD_BF16 else torch.float32
    sc = 1.0 if d.dtype == PD_BF16 else 0.125
    g = torch.Generator().manual_seed(n_sel + Ld)
    r = lambda *s: (torch.randn(s, generator=g) * sc).to(tdt).cuda()
    ks, vs = r(B, Hkv, max(n_sel, 1), D), r(B, Hkv, max(n_sel, 1), D)
    kst, vst = r(B, Lq + 4, Hkv, D), r(B, Lq + 4, Hkv, D)
    dec = random_decode_inputs(d, seed=n_sel, scale=sc)
    o, lse = run_compact(d, n_sel, dec, ks, vs, kst, vst, n_static, splits)
    torch.cuda.synchronize()
    ksh, vsh = h64(ks)[:, :, :n_sel], h64(vs)[:, :, :n_sel]
    qd, kd, vd = (h64(dec[n]) for n in ("q_dec", "k_dec", "v_dec"))
    for b in range(B):
        for h in range(Hq):
            ro, rl = oracle.decode_compact_unit_ref(qd, kd, vd, ksh, vsh, h64(kst), h64(vst), n_static, b, h)
            assert_out_close(d, h64(o[b, :, h]), ro, f"compact decode O (b={b}, h={h})")
            g = h // (Hq // Hkv)
            keys = np.concatenate([ksh[b, g], h64(kst)[b, :n_static, g], kd[b, :, g]])
            assert_lse_close(d, h64(lse[b, h]), rl, qd[b, :, h], keys, f"compact decode LSE (b={b}, h={h})")
