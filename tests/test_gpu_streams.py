"""Calls on different streams, with their own outputs and workspaces, are
independent: the same calls launched concurrently on three streams (two
decodes with different inputs and shard counts, and a prefill into fresh
buffers) give the bits of the sequential run on the default stream."""

import pytest
import torch

from gpu_path import random_decode_inputs, random_prefill_inputs, run_decode, run_prefill, run_select
from paper_2606_10537_amd._lib import PD_BF16, Dims

pytestmark = pytest.mark.gpu


def bits(t):
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


def same(a, b):
    return torch.equal(bits(a), bits(b))


def test_concurrent_streams_match_sequential():
    print("[streams] bf16 B=2 N=4 C=100 H=4/2 d=128", flush=True)
    d = Dims(2, 4, 100, 9, 7, 33, 4, 2, 128, PD_BF16)
    K, Bt = 2, 60
    x = random_prefill_inputs(d, seed=11)
    x2 = random_prefill_inputs(d, seed=12)
    out = run_prefill(d, x)
    dec = [random_decode_inputs(d, seed=13), random_decode_inputs(d, seed=14)]
    sel = [run_select(d, K, Bt, dd["q_dec"], out["key_mean"], out["tok_rank"])[:2] for dd in dec]
    splits = [3, 0]
    torch.cuda.synchronize()

    def decode(i):
        ci, ts = sel[i]
        return run_decode(d, K, Bt, dec[i], out, ci, ts, x["k_qm"], x["v_qm"], d.q_len, num_splits=splits[i])

    ref = [decode(0), decode(1)]
    ref_pre = run_prefill(d, x2)
    torch.cuda.synchronize()

    streams = [torch.cuda.Stream() for _ in range(3)]
    for rep in range(3):
        got = [None, None]
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                got[i] = decode(i)
        with torch.cuda.stream(streams[2]):
            got_pre = run_prefill(d, x2)
        torch.cuda.synchronize()
        for i in range(2):
            assert same(got[i][0], ref[i][0]) and same(got[i][1], ref[i][1]), (rep, i)
        for k in ref_pre:
            assert same(got_pre[k], ref_pre[k]), (rep, k)
