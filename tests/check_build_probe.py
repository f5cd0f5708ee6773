"""Run in its own process by test_gpu_check_build.py: loads the index-checking build libpd_check.so and
feeds the index consumers (gathered decode, bf16 and fp32, with and without Split-S; the static-mode
gather; the full-mask joint gather) one out-of-range kept chunk or slot in one sequence.  That build
replaces such a row by a valid one before reading and writes the dependent outputs as NaN, so every
access stays in bounds.  Prints one JSON object of named checks; exit status 0 iff all hold."""

import json
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

from paper_2606_10537_amd import _lib  # noqa: E402
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims  # noqa: E402

_lib.load(os.path.join(ROOT, "paper_2606_10537_amd", "libpd_check.so"))
import oracle  # noqa: E402
from gpu_path import h64, random_decode_inputs, random_indices, random_prefill_inputs, run_decode, run_prefill  # noqa: E402

checks = {}


def nan_rows(o, b):
    return bool(torch.isnan(o[b].float()).all())


def finite(o, b):
    return bool(torch.isfinite(o[b].float()).all())


for dt in (PD_BF16, PD_FP32):
    d = Dims(2, 4, 64, 8, 8, 32, 4, 2, 128, dt)
    x = random_prefill_inputs(d, seed=5)
    cache = run_prefill(d, x)
    dec = random_decode_inputs(d, seed=6)
    ci, ts = random_indices(d, 2, 16, seed=7)
    for splits in (1, 3):
        tag = f"{'bf16' if dt == PD_BF16 else 'fp32'}/splits{splits}"
        o0, _ = run_decode(d, 2, 16, dec, cache, ci, ts, x["k_qm"], x["v_qm"], 8, splits)
        bad_c = ci.clone()
        bad_c[1, 0] = d.n_chunks                 # chunk index past N in sequence 1
        o1, l1 = run_decode(d, 2, 16, dec, cache, bad_c, ts, x["k_qm"], x["v_qm"], 8, splits)
        bad_s = ts.clone()
        bad_s[0, 1, 3] = 0                       # slot 0 (BOS) listed as a kept token in sequence 0
        bad_s[0, 0, 5] = d.chunk_len + 1         # slot past C
        o2, _ = run_decode(d, 2, 16, dec, cache, ci, bad_s, x["k_qm"], x["v_qm"], 8, splits)
        torch.cuda.synchronize()
        ref, _ = oracle.decode_ref(h64(dec["q_dec"]), h64(dec["k_dec"]), h64(dec["v_dec"]), h64(cache["k_cache"]),
                                   h64(cache["v_cache"]), ci.cpu().numpy(), ts.cpu().numpy(), h64(x["k_qm"]),
                                   h64(x["v_qm"]), 8)
        tol = 1e-2 + (2.0 ** -8 * np.abs(ref) if dt == PD_BF16 else 0) if dt == PD_BF16 else 1e-5
        checks[f"{tag}: valid indices match the oracle"] = bool(np.all(np.abs(h64(o0) - ref) <= tol))
        checks[f"{tag}: bad chunk -> its sequence NaN"] = nan_rows(o1, 1) and bool(torch.isnan(l1[1]).all())
        checks[f"{tag}: bad chunk -> other sequence unchanged"] = bool(torch.equal(o1[0], o0[0]))
        checks[f"{tag}: bad slots -> its sequence NaN"] = nan_rows(o2, 0)
        checks[f"{tag}: bad slots -> other sequence unchanged"] = bool(torch.equal(o2[1], o0[1]))

    # static-mode gather and full-mask joint gather
    n_sel = 2 * 17
    ks = torch.empty((2, d.n_heads_kv, n_sel, 128), dtype=x["k_pre"].dtype, device="cuda")
    vs = torch.empty_like(ks)
    bad_c = ci.clone()
    bad_c[0, 1] = -1
    _lib.pd_gather_selected(d, 2, 16, cache["k_cache"], cache["v_cache"], bad_c, ts, ks, vs)
    Lj = n_sel + d.q_len
    qj = torch.empty((2, Lj, d.n_heads_q, 128), dtype=x["k_pre"].dtype, device="cuda")
    kj = torch.empty((2, Lj, d.n_heads_kv, 128), dtype=x["k_pre"].dtype, device="cuda")
    vj = torch.empty_like(kj)
    _lib.pd_gather_joint(d, 2, 16, bad_c, ts, x["q_pre"], cache["k_cache"], cache["v_cache"], x["q_qm"], x["k_qm"],
                         x["v_qm"], 1e4, qj, kj, vj)
    torch.cuda.synchronize()
    tag = "bf16" if dt == PD_BF16 else "fp32"
    checks[f"{tag}: gather of a bad chunk -> its rows NaN"] = bool(torch.isnan(ks[0, :, 17:34].float()).all())
    checks[f"{tag}: gather -> the rows of good chunks finite"] = (bool(torch.isfinite(ks[0, :, :17].float()).all())
                                                                  and finite(ks, 1))
    checks[f"{tag}: joint gather of a bad chunk -> its rows NaN"] = bool(torch.isnan(kj[0, 17:34].float()).all())
    checks[f"{tag}: joint gather -> other rows finite"] = (bool(torch.isfinite(kj[0, :17].float()).all())
                                                          and bool(torch.isfinite(qj[1].float()).all()))

print(json.dumps(checks))
sys.exit(0 if all(checks.values()) else 1)
