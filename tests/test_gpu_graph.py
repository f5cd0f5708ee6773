"""Stage (b) + (c) of one layer captured in a HIP graph (the per-step launches of
the denoising loop): every replay, with eager launches and synchronisations in
between, gives bit-for-bit the outputs of the same calls made eagerly.  The
library issues kernels only (no memset or copy nodes), so the captured graph
is the plain launch sequence."""

import pytest
import torch

from gpu_path import run_prefill, workspace
from paper_2606_10537_amd import _lib, synth

pytestmark = pytest.mark.gpu


def test_select_decode_graph_replays_match_eager():
    w = synth.WORKLOADS[2]
    d = w.dims()
    x = synth.make_prefill(w, 0, "cuda")
    out = run_prefill(d, x)
    K, Bt = w.top_k, w.tok_budget
    decs = [synth.make_decode(w, 0, t, "cuda") for t in range(2)]
    ci = torch.empty((d.batch, K), dtype=torch.int32, device="cuda")
    ts = torch.empty((d.batch, K, Bt), dtype=torch.int32, device="cuda")
    od = torch.empty_like(decs[0]["q_dec"])
    lse = torch.empty((d.batch, d.n_heads_q, d.dec_len), dtype=torch.float32, device="cuda")
    ws1 = workspace(_lib.pd_workspace_bytes(d, K, Bt, 0, 1))
    ws2 = workspace(_lib.pd_workspace_bytes(d, K, Bt, 0, 2))

    def step(dec, stream):
        _lib.pd_score_select(d, K, Bt, dec["q_dec"], out["key_mean"], out["tok_rank"], ci, ts, None, ws1, stream)
        _lib.pd_sparse_decode_attn(d, K, Bt, dec["q_dec"], dec["k_dec"], dec["v_dec"], out["k_cache"],
                                   out["v_cache"], ci, ts, x["k_qm"], x["v_qm"], w.q_len, od, lse, 0, ws2, stream)

    ref = []
    for dec in decs:
        step(dec, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        ref.append((ci.clone(), ts.clone(), od.clone(), lse.clone()))

    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            step(decs[1], torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    for replay in range(3):
        step(decs[0], torch.cuda.current_stream().cuda_stream)       # eager work between replays
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip((ci, ts, od, lse), ref[0]))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((ci, ts, od, lse), ref[1]):
            assert torch.equal(a, b), f"replay {replay} differs from the eager result"
