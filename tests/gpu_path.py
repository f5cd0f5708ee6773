"""Test helpers: run each stage through the C ABI, copy results to host, rule A.

Outputs are pre-filled with NaN (float) or -1 (int) so that an element the
kernels fail to write shows up as a mismatch.
"""

import numpy as np
import torch

from paper_2606_10537_amd import _lib
from paper_2606_10537_amd._lib import PD_BF16, Dims


def h64(t):
    """Exact host float64 copy of a device tensor (bf16 and fp32 upcast exactly)."""
    return t.detach().float().cpu().double().numpy()


def torch_dtype(d: Dims):
    return torch.bfloat16 if d.dtype == PD_BF16 else torch.float32


def workspace(nbytes, device="cuda"):
    """Caller-owned scratch (zero-filled, so that a stale value never passes for a result)."""
    return torch.zeros(max(nbytes, 16), dtype=torch.uint8, device=device)


def run_prefill(d: Dims, x, stream=None, chunk_score=False):
    dev, dt = x["q_pre"].device, x["q_pre"].dtype
    B, N, C, Hq, Hkv, D = d.batch, d.n_chunks, d.chunk_len, d.n_heads_q, d.n_heads_kv, d.head_dim
    odt = torch.float32 if d.out_fp32 else dt
    out = {
        "o": torch.full((B, N, d.seq_len, Hq, D), float("nan"), dtype=odt, device=dev),
        "k_cache": torch.full((B, N, Hkv, C + 1, D), float("nan"), dtype=dt, device=dev),
        "v_cache": torch.full((B, N, Hkv, C + 1, D), float("nan"), dtype=dt, device=dev),
        "tok_score": torch.full((B, N, C), float("nan"), dtype=torch.float32, device=dev),
        "tok_rank": torch.full((B, N, C), -1, dtype=torch.int32, device=dev),
        "key_mean": torch.full((B, N, Hkv, D), float("nan"), dtype=torch.float32, device=dev),
    }
    if chunk_score:
        out["chunk_score"] = torch.full((B, N), float("nan"), dtype=torch.float32, device=dev)
    ws = workspace(_lib.pd_workspace_bytes(d, which=0), dev)
    _lib.pd_prefill_chunks(d, x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"],
                           out["o"], out["k_cache"], out["v_cache"], out["tok_score"], out["tok_rank"],
                           out["key_mean"], ws, stream, chunk_score=out.get("chunk_score"))
    return out


def run_select(d: Dims, top_k, tok_budget, q_dec, key_mean, tok_rank, stream=None):
    dev = q_dec.device
    ci = torch.full((d.batch, top_k), -1, dtype=torch.int32, device=dev)
    ts = torch.full((d.batch, top_k, tok_budget), -1, dtype=torch.int32, device=dev)
    cs = torch.full((d.batch, d.n_chunks), float("nan"), dtype=torch.float32, device=dev)
    ws = workspace(_lib.pd_workspace_bytes(d, top_k, tok_budget, 0, 1), dev)
    _lib.pd_score_select(d, top_k, tok_budget, q_dec, key_mean, tok_rank, ci, ts, cs, ws, stream)
    return ci, ts, cs


def run_decode(d: Dims, top_k, tok_budget, dec, cache, ci, ts, k_static, v_static, n_static, num_splits=0,
               with_lse=True, stream=None):
    dev = dec["q_dec"].device
    odt = torch.float32 if d.out_fp32 else dec["q_dec"].dtype
    o = torch.full(dec["q_dec"].shape, float("nan"), dtype=odt, device=dev)
    lse = (torch.full((d.batch, d.n_heads_q, d.dec_len), float("nan"), dtype=torch.float32, device=dev)
           if with_lse else None)
    ws = workspace(_lib.pd_workspace_bytes(d, top_k, tok_budget, num_splits, 2), dev)
    _lib.pd_sparse_decode_attn(d, top_k, tok_budget, dec["q_dec"], dec["k_dec"], dec["v_dec"],
                               cache["k_cache"], cache["v_cache"], ci, ts, k_static, v_static, n_static, o,
                               lse, num_splits, ws, stream)
    return o, lse


def random_prefill_inputs(d: Dims, seed, device="cuda", scale=1.0):
    """Seeded i.i.d. N(0, scale^2) inputs in the library layouts (rounded to the element type)."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    B, N, C1, Hq, Hkv, D = d.batch, d.n_chunks, d.chunk_len + 1, d.n_heads_q, d.n_heads_kv, d.head_dim
    Lqm = d.q_len + d.m_len
    qm = (B, N, Lqm) if d.qm_per_chunk else (B, Lqm)
    dt = torch_dtype(d)
    r = lambda *s: (torch.randn(s, generator=g) * scale).to(dt).to(device)
    return {"q_pre": r(B, N, C1, Hq, D), "k_pre": r(B, N, C1, Hkv, D), "v_pre": r(B, N, C1, Hkv, D),
            "q_qm": r(*qm, Hq, D), "k_qm": r(*qm, Hkv, D), "v_qm": r(*qm, Hkv, D)}


def random_decode_inputs(d: Dims, seed, device="cuda", scale=1.0):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    dt = torch_dtype(d)
    r = lambda *s: (torch.randn(s, generator=g) * scale).to(dt).to(device)
    B, Ld, Hq, Hkv, D = d.batch, d.dec_len, d.n_heads_q, d.n_heads_kv, d.head_dim
    return {"q_dec": r(B, Ld, Hq, D), "k_dec": r(B, Ld, Hkv, D), "v_dec": r(B, Ld, Hkv, D)}


def random_indices(d: Dims, top_k, tok_budget, seed, device="cuda"):
    """Valid selections: distinct ascending chunks and distinct ascending slots in 1..C."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    ci = torch.stack([torch.sort(torch.randperm(d.n_chunks, generator=g)[:top_k])[0] for _ in range(d.batch)])
    ts = torch.stack([torch.stack([torch.sort(torch.randperm(d.chunk_len, generator=g)[:tok_budget] + 1)[0]
                                   for _ in range(top_k)]) for _ in range(d.batch)])
    return ci.to(torch.int32).to(device), ts.to(torch.int32).to(device)


def check_topk_rule_a(x, got, k, band=1e-3):
    """Rule A: the GPU set has k distinct members in ascending order, contains every
    element the oracle pins in (score above the (k+1)-th by more than `band`) and no
    element it pins out.  Returns the number of unpinned elements."""
    x = np.asarray(x, dtype=np.float64)
    got = np.asarray(got)
    n = x.shape[0]
    assert got.shape == (k,), (got.shape, k)
    assert np.all(np.diff(got) > 0), f"not strictly ascending: {got}"
    assert got.min() >= 0 and got.max() < n
    srt = np.sort(x)[::-1]
    tau = srt[k - 1]
    sig = srt[k] if k < n else -np.inf
    pin_in = (x >= tau) & (x - sig > band)
    pin_out = (x <= sig) & (tau - x > band)
    gs = set(got.tolist())
    missing = [i for i in np.nonzero(pin_in)[0] if i not in gs]
    extra = [i for i in np.nonzero(pin_out)[0] if i in gs]
    assert not missing and not extra, f"rule A violated: missing {missing} extra {extra}"
    return int(n - pin_in.sum() - pin_out.sum())


def check_rank_consistent(e_ref, rank, band=1e-3):
    """GPU token ranks of one chunk: a permutation of 0..C-1 that orders every pair
    whose oracle scores differ by more than `band` the same way as the oracle."""
    e_ref = np.asarray(e_ref, dtype=np.float64)
    rank = np.asarray(rank)
    C = e_ref.shape[0]
    assert np.array_equal(np.sort(rank), np.arange(C)), "ranks are not a permutation"
    before = rank[:, None] < rank[None, :]            # i ranked before j
    bad = before & (e_ref[None, :] - e_ref[:, None] > band)
    assert not bad.any(), f"{int(bad.sum())} pairs ranked against the oracle's order"
