"""GPU parity at the size limits the C ABI accepts, against the oracle.

* Prefill at the largest chunk length (C = 4096): every head's output, the
  cache bits, the key means and the Eq. 5 scores, bf16 and fp32, with GQA.
* Decode over a kept prefix longer than the decode kernel's row table (2048
  rows per shard): two whole chunks of 4096 tokens kept (8194 prefix rows), so
  the library must cut the KV rows into several shards whatever the caller
  asks; the per-step (gathered) and the compact entry points, automatic and
  explicit shard counts.

Tolerances as in test_gpu_parity (output bound, LSE bound); the decode's
cache is built from the inputs by a layout permutation, not by the prefill.
"""

import numpy as np
import pytest
import torch

from gpu_path import h64, random_decode_inputs, random_prefill_inputs, run_decode, run_prefill, workspace
from paper_2606_10537_amd import _lib
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims
from test_gpu_parity import decode_check, prefill_units_check

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dt", [PD_BF16, PD_FP32])
def test_prefill_max_chunk_len(dt):
    d = Dims(1, 2, 4096, 8, 3, 8, 2, 1, 128, dt)
    print(f"[limits] prefill C=4096 dtype={dt}", flush=True)
    x = random_prefill_inputs(d, seed=4096 + dt, scale=1.0 if dt == PD_BF16 else 0.125)
    out = run_prefill(d, x)
    torch.cuda.synchronize()
    prefill_units_check(d, x, out, [(0, 0), (0, 1)])


def cache_of(t):
    """Chunk rows [B][N][1+C][H][d] -> cache layout [B][N][H][1+C][d] (torch permutation)."""
    return t.permute(0, 1, 3, 2, 4).contiguous()


@pytest.mark.parametrize("num_splits", [0, 1, 9])
def test_decode_prefix_beyond_row_table(num_splits):
    """8194 kept rows: more than one shard's row table; the gathered decode against the oracle."""
    d = Dims(1, 2, 4096, 8, 0, 16, 2, 1, 128, PD_BF16)
    K, Bt = 2, 4096
    print(f"[limits] decode n_sel={K * (1 + Bt)} num_splits={num_splits}", flush=True)
    x = random_prefill_inputs(d, seed=77)
    cache = {"k_cache": cache_of(x["k_pre"]), "v_cache": cache_of(x["v_pre"])}
    dec = random_decode_inputs(d, seed=78)
    ci = torch.tensor([[0, 1]], dtype=torch.int32, device="cuda")
    ts = torch.arange(1, Bt + 1, dtype=torch.int32, device="cuda").repeat(1, K, 1)
    splits = _lib.pd_decode_splits(d, K, Bt, d.q_len, num_splits)
    assert splits >= 5, splits   # ceil(8218 rows / 64) tiles, at most 32 tiles per shard
    o, lse = run_decode(d, K, Bt, dec, cache, ci, ts, x["k_qm"], x["v_qm"], d.q_len, num_splits=num_splits)
    torch.cuda.synchronize()
    decode_check(d, K, Bt, dec, cache, ci, ts, x["k_qm"], x["v_qm"], d.q_len, o, lse)


def test_compact_prefix_beyond_row_table():
    """The compact entry point over 8194 prefix rows equals the gathered decode bit for bit."""
    d = Dims(1, 2, 4096, 8, 0, 16, 2, 1, 128, PD_BF16)
    K, Bt = 2, 4096
    n_sel = K * (1 + Bt)
    x = random_prefill_inputs(d, seed=79)
    cache = {"k_cache": cache_of(x["k_pre"]), "v_cache": cache_of(x["v_pre"])}
    dec = random_decode_inputs(d, seed=80)
    ci = torch.tensor([[0, 1]], dtype=torch.int32, device="cuda")
    ts = torch.arange(1, Bt + 1, dtype=torch.int32, device="cuda").repeat(1, K, 1)
    o_g, l_g = run_decode(d, K, Bt, dec, cache, ci, ts, x["k_qm"], x["v_qm"], d.q_len)
    # Contiguous prefix [B][H_kv][n_sel][d]: each chunk's BOS then every slot, i.e. the whole cache rows.
    ks = cache["k_cache"].reshape(1, 2 * (1 + Bt), 1, 128).permute(0, 2, 1, 3).contiguous()
    vs = cache["v_cache"].reshape(1, 2 * (1 + Bt), 1, 128).permute(0, 2, 1, 3).contiguous()
    o = torch.full_like(dec["q_dec"], float("nan"))
    lse = torch.full((1, 2, 16), float("nan"), dtype=torch.float32, device="cuda")
    ws = workspace(_lib.pd_compact_workspace_bytes(d, n_sel, 0))
    _lib.pd_sparse_decode_attn_compact(d, n_sel, dec["q_dec"], dec["k_dec"], dec["v_dec"], ks, vs, x["k_qm"],
                                       x["v_qm"], d.q_len, o, lse, 0, ws)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o_g.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), l_g.view(torch.int32))
