"""Seeded synthetic inputs shaped like the paper's 8K-32K workloads.

This module only draws random tensors (torch, on any device) and places them
in the library's layouts; it holds none of the method's arithmetic.  The HIP
path and the CPU oracle both receive exactly these tensors (the oracle as a
host float64 copy).

Recipe (stands in for LongBench / InfiniteBench prompts on a 7B dLLM; no
dataset content is used -- only the workload shapes of Sections 6.3 and
Appendix A: C = 1024, K of 2-4, B of 256-512, d = 128, GQA):

* Q/K/V entries i.i.d. N(0, 1) * sigma, rounded to the call's element type
  (round-to-nearest-even for bf16).  sigma = 1/8 (= 1/sqrt(64)) for the tiny
  fp32 workload, 1 otherwise.
* The BOS row (chunk slot 0) is one vector per (layer, head), shared by every
  chunk, as the same token at reset position 0 would be.
* The query/pseudo-label rows are one tensor shared by all chunks.
* Planted relevance (workloads with `plant` > 0): per KV head g a random unit
  direction u_g; the content keys of each planted chunk get + alpha*u_g, a
  32-token "needle" span inside it another + alpha*u_g, and the L_q query rows'
  queries and every decode query get + beta*u_{g(h)}.
* Heavy-tailed key norms (`key_lognormal` > 0): every key row (prefix, BOS,
  query/pseudo-label, decode) is scaled by exp(sigma_k * z), z ~ N(0, 1) drawn
  per token and shared across heads.
* Decode rows are drawn fresh for every (layer, step).
"""

import zlib
from dataclasses import dataclass, field

import torch

from ._lib import PD_BF16, PD_FP32, Dims


@dataclass(frozen=True)
class Workload:
    name: str
    cid: int
    batch: int
    n_chunks: int
    chunk_len: int
    q_len: int
    m_len: int
    dec_len: int
    n_heads_q: int
    n_heads_kv: int
    head_dim: int
    top_k: int
    tok_budget: int
    steps: int
    layers: int = 1
    dtype: int = PD_BF16
    sigma: float = 1.0
    plant: int = 0            # number of planted chunks
    plant_stratified: bool = False
    alpha: float = 0.0        # key plant amplitude
    beta: float = 0.0         # query plant amplitude
    key_lognormal: float = 0.0

    def dims(self, batch=None) -> Dims:
        return Dims(batch or self.batch, self.n_chunks, self.chunk_len, self.q_len, self.m_len,
                    self.dec_len, self.n_heads_q, self.n_heads_kv, self.head_dim, self.dtype)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == PD_BF16 else torch.float32

    @property
    def context(self):
        return self.n_chunks * self.chunk_len


_SQ = 128 ** 0.5 * 0.5   # alpha = 0.5 * sqrt(d) for d = 128

WORKLOADS = {
    1: Workload("tiny-fp32", 1, 1, 4, 128, 16, 32, 32, 4, 4, 64, 2, 128, 4, dtype=PD_FP32,
                sigma=1 / 8, plant=1, alpha=0.5, beta=0.5),
    2: Workload("8k-mha", 2, 1, 8, 1024, 64, 256, 256, 32, 32, 128, 2, 512, 64,
                plant=2, alpha=_SQ, beta=_SQ),
    3: Workload("16k-gqa", 3, 1, 16, 1024, 64, 256, 256, 28, 4, 128, 4, 256, 64,
                plant=4, plant_stratified=True, alpha=_SQ, beta=_SQ),
    4: Workload("32k-b4", 4, 4, 32, 1024, 128, 512, 512, 32, 32, 128, 4, 256, 128, key_lognormal=0.3),
    5: Workload("32k-32layer-b8", 5, 8, 32, 1024, 128, 512, 512, 32, 32, 128, 4, 256, 256, layers=32,
                key_lognormal=0.3),
}


def seed_of(w: Workload, *parts) -> int:
    key = "/".join(str(p) for p in (w.cid, *parts))
    return (20260 + w.cid) * 1_000_003 + zlib.crc32(key.encode())


def _gen(w, device, *parts):
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(w, *parts))
    return g


def _randn(shape, g, device):
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def plant_info(w: Workload, layer: int, device="cpu"):
    """Planted chunk indices (B, plant), needle offsets and unit directions (Hkv, d)."""
    if w.plant == 0:
        return None
    g = _gen(w, "cpu", layer, "plant")
    chunks = []
    for b in range(w.batch):
        if w.plant_stratified:
            per = w.n_chunks // w.plant
            sel = [i * per + int(torch.randint(per, (1,), generator=g)) for i in range(w.plant)]
        else:
            sel = sorted(torch.randperm(w.n_chunks, generator=g)[: w.plant].tolist())
        chunks.append(sel)
    span = min(32, w.chunk_len)
    needles = torch.randint(0, w.chunk_len - span + 1, (w.batch, w.plant), generator=g)
    u = torch.randn((w.n_heads_kv, w.head_dim), generator=g)
    u = u / u.norm(dim=1, keepdim=True)
    return {"chunks": chunks, "needles": needles.tolist(), "span": span, "u": u.to(device)}


def _key_scale(shape_tokens, g, device, sig):
    return torch.exp(sig * _randn(shape_tokens, g, device))


def make_prefill(w: Workload, layer: int = 0, device="cpu", batch=None):
    """Stage (a) inputs of one layer in the library layouts (see include/pd.h)."""
    B = batch or w.batch
    N, C1, Hq, Hkv, d = w.n_chunks, w.chunk_len + 1, w.n_heads_q, w.n_heads_kv, w.head_dim
    Lqm = w.q_len + w.m_len
    out = {}
    for name, H in (("q", Hq), ("k", Hkv), ("v", Hkv)):
        g = _gen(w, device, layer, name + "_pre")
        x = _randn((B, N, C1, H, d), g, device) * w.sigma
        bos = _randn((H, d), _gen(w, device, layer, name + "_bos"), device) * w.sigma
        x[:, :, 0] = bos
        qm = _randn((B, Lqm, H, d), _gen(w, device, layer, name + "_qm"), device) * w.sigma
        out[name + "_pre"], out[name + "_qm"] = x, qm
    if w.key_lognormal > 0:
        g = _gen(w, device, layer, "key_norms")
        out["k_pre"] *= _key_scale((B, N, C1, 1, 1), g, device, w.key_lognormal)
        out["k_qm"] *= _key_scale((B, Lqm, 1, 1), g, device, w.key_lognormal)
    pl = plant_info(w, layer, device)
    if pl is not None:
        u = pl["u"]
        G = Hq // Hkv
        for b in range(B):
            for i, n in enumerate(pl["chunks"][b % w.batch]):
                out["k_pre"][b, n, 1:] += w.alpha * u
                o = pl["needles"][b % w.batch][i]
                out["k_pre"][b, n, 1 + o: 1 + o + pl["span"]] += w.alpha * u
        out["q_qm"][:, : w.q_len] += w.beta * u.repeat_interleave(G, dim=0)
    return {k: v.to(w.torch_dtype).contiguous() for k, v in out.items()}


def make_decode(w: Workload, layer: int = 0, step: int = 0, device="cpu", batch=None):
    """Stage (b)/(c) per-step inputs: q_dec (B, Ld, Hq, d), k_dec / v_dec (B, Ld, Hkv, d)."""
    B = batch or w.batch
    Ld, Hq, Hkv, d = w.dec_len, w.n_heads_q, w.n_heads_kv, w.head_dim
    out = {
        "q_dec": _randn((B, Ld, Hq, d), _gen(w, device, layer, step, "q_dec"), device) * w.sigma,
        "k_dec": _randn((B, Ld, Hkv, d), _gen(w, device, layer, step, "k_dec"), device) * w.sigma,
        "v_dec": _randn((B, Ld, Hkv, d), _gen(w, device, layer, step, "v_dec"), device) * w.sigma,
    }
    if w.key_lognormal > 0:
        out["k_dec"] *= _key_scale((B, Ld, 1, 1), _gen(w, device, layer, step, "dec_norms"), device,
                                   w.key_lognormal)
    pl = plant_info(w, layer, device)
    if pl is not None:
        out["q_dec"] += w.beta * pl["u"].repeat_interleave(Hq // Hkv, dim=0)
    return {k: v.to(w.torch_dtype).contiguous() for k, v in out.items()}
