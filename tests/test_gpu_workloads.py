"""GPU parity on the five benchmark workloads, in the launch configuration bench.py times.

Workload 1 (tiny, fp32) is checked in full.  The bf16 workloads run one layer at
their real sizes; the oracle checks sampled units: prefill O / cache / key means
/ Eq. 5 scores / token ranks of listed (sequence, chunk) pairs over every head,
chunk selection of every sequence at several steps (rule A), the token sets of
the kept chunks of one sequence (rule A against the oracle's Eq. 5 scores), and
decode outputs of listed (sequence, head) pairs with the oracle run on the
GPU's own indices.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_path import check_rank_consistent, check_topk_rule_a, h64, run_decode, run_prefill, run_select
from paper_2606_10537_amd import synth
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32
from test_gpu_parity import decode_check, prefill_units_check

pytestmark = pytest.mark.gpu


def run_workload(wid, batch=None, steps=(0,), prefill_units=(), decode_units=(), token_check_b=0,
                 full=False, out_fp32=0):
    w = synth.WORKLOADS[wid]
    d = w.dims(batch)
    d.out_fp32 = out_fp32
    x = synth.make_prefill(w, 0, "cuda", batch=batch)
    out = run_prefill(d, x)
    torch.cuda.synchronize()
    B = d.batch
    if full:
        prefill_units = [(b, n) for b in range(B) for n in range(d.n_chunks)]
    print(f"[workload {wid}] prefill done; checking {len(prefill_units)} units", flush=True)
    prefill_units_check(d, x, out, prefill_units)

    # Oracle key means of every chunk, one (b, n) slice at a time.
    km_ref = np.zeros((B, d.n_chunks, d.n_heads_kv, d.head_dim))
    for b in range(B):
        for n in range(d.n_chunks):
            km_ref[b, n] = oracle.key_mean_ref(h64(x["k_pre"][b:b + 1, n:n + 1]))[0, 0]
    unpinned = 0
    for t in steps:
        dec = synth.make_decode(w, 0, t, "cuda", batch=batch)
        ci, tsl, cs = run_select(d, w.top_k, w.tok_budget, dec["q_dec"], out["key_mean"], out["tok_rank"])
        o, lse = run_decode(d, w.top_k, w.tok_budget, dec, out, ci, tsl, x["k_qm"], x["v_qm"], w.q_len)
        torch.cuda.synchronize()
        s_ref = oracle.chunk_scores_ref(h64(dec["q_dec"]), km_ref)
        np.testing.assert_allclose(h64(cs), s_ref, rtol=1e-4, atol=1e-4)
        for b in range(B):
            unpinned += check_topk_rule_a(s_ref[b], ci[b].cpu().numpy(), w.top_k)
        assert np.array_equal(tsl.cpu().numpy(),
                              oracle.tokens_by_rank_ref(out["tok_rank"].cpu().numpy(), ci.cpu().numpy(), w.tok_budget))
        if t == steps[0] and token_check_b is not None:
            b = token_check_b
            for kk, n in enumerate(ci[b].cpu().tolist()):
                xs = {k: h64(v[b:b + 1, n:n + 1] if k.endswith("_pre") else v[b:b + 1]) for k, v in x.items()}
                e = np.zeros(d.chunk_len)
                for h in range(d.n_heads_q):
                    e += oracle.prefill_unit_ref(xs["q_pre"], xs["k_pre"], xs["v_pre"], xs["q_qm"], xs["k_qm"],
                                                 xs["v_qm"], 0, 0, h, d.q_len)["e_head"]
                unpinned += check_topk_rule_a(e, tsl[b, kk].cpu().numpy() - 1, w.tok_budget)
        units = decode_units if decode_units else [(b, h) for b in range(B) for h in range(d.n_heads_q)]
        for b in sorted({u[0] for u in units}):
            decode_check(d, w.top_k, w.tok_budget, dec, out, ci, tsl, x["k_qm"], x["v_qm"], w.q_len, o, lse,
                         heads=[u[1] for u in units if u[0] == b], batches=[b])
        print(f"[workload {wid}] step {t} ok", flush=True)
    print(f"[workload {wid}] unpinned selections within the 1e-3 band: {unpinned}", flush=True)
    return out, x


def test_workload1_tiny_fp32_full():
    w = synth.WORKLOADS[1]
    out, x = run_workload(1, steps=tuple(range(w.steps)), full=True)
    # The planted chunk is recovered at every step (sanity of the synthetic plant, not parity).
    pl = synth.plant_info(w, 0)
    d = w.dims()
    for t in range(w.steps):
        dec = synth.make_decode(w, 0, t, "cuda")
        ci, _, _ = run_select(d, w.top_k, w.tok_budget, dec["q_dec"], out["key_mean"], out["tok_rank"])
        assert pl["chunks"][0][0] in ci[0].cpu().tolist()


def test_workload2_8k():
    run_workload(2, steps=(0, 63), prefill_units=[(0, 0), (0, 7)],
                 decode_units=[(0, 0), (0, 17), (0, 31)])


def test_workload3_16k_gqa():
    run_workload(3, steps=(0, 63), prefill_units=[(0, 3), (0, 15)],
                 decode_units=[(0, 0), (0, 6), (0, 7), (0, 27)])


@pytest.mark.parametrize("out_fp32", [1, 0])
def test_workload4_32k_b4(out_fp32):
    run_workload(4, steps=(0, 127), prefill_units=[(0, 0), (3, 31)],
                 decode_units=[(0, 0), (0, 31), (3, 5)], out_fp32=out_fp32)


def test_workload5_32k_layer_b8():
    """One layer of the 32-layer batch-8 workload (the per-layer launches bench.py times)."""
    run_workload(5, steps=(0, 255), prefill_units=[(7, 17)], decode_units=[(0, 3), (7, 30)], token_check_b=7,
                 out_fp32=1)
