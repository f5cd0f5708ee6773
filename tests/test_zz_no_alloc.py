"""The selection entry point that allocates nothing (scratch in the library's static per-GPU array)
against the workspace entry point on the same inputs: two calls in a row, the second with a smaller
input, then a third with K > N/2.  Indices must be bit-identical (integer work) and the chunk scores
identical (the same kernels run the same fp32 arithmetic in the same order)."""

import numpy as np
import pytest
import torch

from gpu_path import workspace
from paper_2606_10537_amd import _lib
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims

pytestmark = pytest.mark.gpu


def inputs(d, seed):
    g = torch.Generator().manual_seed(seed)
    dt = torch.bfloat16 if d.dtype == PD_BF16 else torch.float32
    q = torch.randn((d.batch, d.dec_len, d.n_heads_q, d.head_dim), generator=g).to(dt).cuda()
    km = torch.randn((d.batch, d.n_chunks, d.n_heads_kv, d.head_dim), generator=g).cuda()
    rank = torch.argsort(torch.rand((d.batch, d.n_chunks, d.chunk_len), generator=g), dim=2).to(torch.int32).cuda()
    return q, km, rank


def outputs(d, K, Bt):
    return (torch.full((d.batch, K), -1, dtype=torch.int32, device="cuda"),
            torch.full((d.batch, K, Bt), -1, dtype=torch.int32, device="cuda"),
            torch.full((d.batch, d.n_chunks), float("nan"), dtype=torch.float32, device="cuda"))


CALLS = [
    # (dims, K, B_tok): the 32K batch-8 per-layer shape, then smaller ones
    (Dims(8, 32, 1024, 128, 512, 512, 32, 32, 128, PD_BF16), 4, 256),
    (Dims(2, 8, 300, 16, 8, 40, 8, 2, 64, PD_FP32), 3, 100),
    (Dims(1, 100, 40, 4, 0, 20, 4, 2, 64, PD_BF16), 80, 9),
]


def test_noalloc_select_matches_workspace_select():
    for i, (d, K, Bt) in enumerate(CALLS):
        print(f"[no-alloc] call {i}: B={d.batch} N={d.n_chunks} C={d.chunk_len} L_d={d.dec_len} K={K}", flush=True)
        q, km, rank = inputs(d, 100 + i)
        ci0, ts0, cs0 = outputs(d, K, Bt)
        ws = workspace(_lib.pd_workspace_bytes(d, K, Bt, 0, 1))
        _lib.pd_score_select(d, K, Bt, q, km, rank, ci0, ts0, cs0, ws)
        ci1, ts1, cs1 = outputs(d, K, Bt)
        _lib.pd_score_select_noalloc(d, K, Bt, q, km, rank, ci1, ts1, cs1)
        torch.cuda.synchronize()
        assert torch.equal(ci1, ci0), f"call {i}: chunk_idx"
        assert torch.equal(ts1, ts0), f"call {i}: tok_slot"
        assert np.array_equal(cs1.cpu().numpy().view(np.int32), cs0.cpu().numpy().view(np.int32)), f"call {i}: scores"
        assert (ci1 >= 0).all() and (ts1 >= 1).all()


def test_noalloc_select_rejects_oversize():
    d = Dims(64, 1024, 64, 4, 0, 512, 64, 8, 128, PD_BF16)
    q = torch.zeros(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(_lib.PdError) as e:
        _lib.pd_score_select_noalloc(d, 4, 8, q, q, q, q, q)
    assert e.value.status == 2 and "scratch" in str(e.value)
