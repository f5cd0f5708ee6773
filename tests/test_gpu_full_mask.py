"""GPU parity of the full-mask cache construction against the oracle's
full-mask module, through the C ABI: pd_gather_joint (joint rows at
continuous positions), the dense joint attention over them and the decoding
steps over the joint prefix (both pd_sparse_decode_attn_compact).

Tolerances.
* rope_base = 0: the joint rows are copies of input rows: bit-exact, and the
  prefix-layout copies bit-identical to the decode-layout rows.
* rotated Q and K: the kernel evaluates the rotation in double and rounds once
  (through fp32) to the element type, so it is within half an ulp of the
  oracle's fp64 value: |got - ref| <= 2^-8 |ref| (bf16) or 2^-24 |ref| (fp32),
  each with 2^-24 |ref| more for the fp32 step and 1e-10 max|x| for the angle's
  double rounding (angles up to about 4e4 rad).
* joint attention and decoding: the decode output bound (1e-2 max-abs for bf16
  inputs, 1e-5 for fp32, plus the bf16 output rounding) and the decode LSE
  bound (log(1 + 2^-8) for the bf16 weights plus the logits' fp32 error, per
  row; 1e-4 for fp32).  The oracle attends over its own joint rows rounded to
  the element type (RNE on the host), never over the kernel's.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_path import h64, random_decode_inputs, random_indices, random_prefill_inputs, run_prefill, workspace
from paper_2606_10537_amd import _lib, synth
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims
from test_gpu_parity import assert_lse_close, assert_out_close, bits

pytestmark = pytest.mark.gpu


def run_joint(d, K, Bt, ci, ts, x, k_cache, v_cache, base, pref=True):
    Lj = K * (1 + Bt) + d.q_len
    dt = x["q_pre"].dtype
    nan = lambda *s: torch.full(s, float("nan"), dtype=dt, device="cuda")
    B, Hq, Hkv, D = d.batch, d.n_heads_q, d.n_heads_kv, d.head_dim
    out = {"q": nan(B, Lj, Hq, D), "k": nan(B, Lj, Hkv, D), "v": nan(B, Lj, Hkv, D)}
    if pref:
        out["kp"], out["vp"] = nan(B, Hkv, Lj, D), nan(B, Hkv, Lj, D)
    _lib.pd_gather_joint(d, K, Bt, ci, ts, x["q_pre"], k_cache, v_cache, x["q_qm"], x["k_qm"], x["v_qm"], base,
                         out["q"], out["k"], out["v"], out.get("kp"), out.get("vp"))
    return out


def joint_dims(d, Lj):
    return Dims(d.batch, d.n_chunks, d.chunk_len, d.q_len, d.m_len, Lj, d.n_heads_q, d.n_heads_kv, d.head_dim,
                d.dtype, d.sm_scale, d.qm_per_chunk)


def run_dense(dj, q, k, v, num_splits=0):
    """The joint pass: compact decode with no prefix and the L_j joint rows as its own rows."""
    o = torch.full(q.shape, float("nan"), dtype=q.dtype, device="cuda")
    lse = torch.full((dj.batch, dj.n_heads_q, dj.dec_len), float("nan"), dtype=torch.float32, device="cuda")
    ws = workspace(_lib.pd_compact_workspace_bytes(dj, 0, num_splits))
    _lib.pd_sparse_decode_attn_compact(dj, 0, q, k, v, None, None, None, None, 0, o, lse, num_splits, ws)
    return o, lse


def run_steps(d, n_sel, dec, kp, vp, num_splits=0):
    o = torch.full(dec["q_dec"].shape, float("nan"), dtype=dec["q_dec"].dtype, device="cuda")
    lse = torch.full((d.batch, d.n_heads_q, d.dec_len), float("nan"), dtype=torch.float32, device="cuda")
    ws = workspace(_lib.pd_compact_workspace_bytes(d, n_sel, num_splits))
    _lib.pd_sparse_decode_attn_compact(d, n_sel, dec["q_dec"], dec["k_dec"], dec["v_dec"], kp, vp, None, None, 0,
                                       o, lse, num_splits, ws)
    return o, lse


def cache_layout(t):
    """Chunk rows [B][N][1+C][H][d] -> cache layout [B][N][H][1+C][d]."""
    return t.permute(0, 1, 3, 2, 4).contiguous()


def round_to(a, dtype):
    """fp64 host array rounded to the element type (RNE), back as fp64."""
    return torch.from_numpy(np.ascontiguousarray(a)).to(dtype).double().numpy()


def assert_rotated_close(d, got, ref, xmax, what):
    rel = (2.0 ** -8 if d.dtype == PD_BF16 else 2.0 ** -24) + 2.0 ** -24
    err = np.abs(got - ref)
    bound = rel * np.abs(ref) + 1e-10 * xmax
    worst = np.max(err - bound)
    assert worst <= 0, f"{what}: max-abs {err.max():.3g} exceeds the bound by {worst:.3g}"


def check_rows(d, out, ref, base, xmax, what):
    """Joint rows of one tensor against the oracle: bits when base = 0, else half an ulp."""
    if base == 0:
        assert np.array_equal(h64(out), ref), f"{what}: not a bit-exact copy"
    else:
        assert_rotated_close(d, h64(out), ref, xmax, what)


CASES = [
    # dtype, B, N, C, Lq, Lm, Hq, Hkv, D, K, Bt, per_chunk, base
    (PD_BF16, 2, 5, 64, 16, 8, 4, 2, 128, 3, 10, 0, 0.0),
    (PD_BF16, 2, 5, 64, 16, 8, 4, 2, 128, 3, 10, 0, 10000.0),
    (PD_BF16, 1, 4, 300, 33, 0, 8, 8, 64, 4, 300, 1, 500000.0),   # every chunk and token kept
    (PD_BF16, 1, 1, 1, 1, 1, 1, 1, 128, 1, 1, 0, 10000.0),         # smallest
    (PD_FP32, 2, 3, 77, 9, 3, 4, 1, 128, 2, 5, 1, 10000.0),
    (PD_FP32, 1, 2, 16, 4, 4, 2, 2, 64, 1, 1, 0, 0.0),             # K = 1: query rows not moved
]


@pytest.mark.parametrize("case", CASES, ids=[str(c) for c in CASES])
def test_gather_joint_parity(case):
    """Joint Q, K, V of every row against the oracle; the prefix-layout copies
    bit-identical to the decode-layout K, V; every element written."""
    dt, B, N, C, Lq, Lm, Hq, Hkv, D, K, Bt, pc, base = case
    d = Dims(B, N, C, Lq, Lm, 8, Hq, Hkv, D, dt, 0.0, pc)
    print(f"[gather joint] {case}", flush=True)
    x = random_prefill_inputs(d, seed=sum(case[1:12]), scale=1.0 if dt == PD_BF16 else 0.25)
    kc, vc = cache_layout(x["k_pre"]), cache_layout(x["v_pre"])
    ci, ts = random_indices(d, K, Bt, seed=K * 7 + Bt)
    out = run_joint(d, K, Bt, ci, ts, x, kc, vc, base)
    torch.cuda.synchronize()
    rq, rk, rv = oracle.joint_rows_ref(h64(x["q_pre"]), h64(kc), h64(vc), h64(x["q_qm"]), h64(x["k_qm"]),
                                       h64(x["v_qm"]), ci.cpu().numpy(), ts.cpu().numpy(), Lq, base)
    xmax = max(float(np.abs(h64(t)).max()) for t in x.values())
    check_rows(d, out["q"], rq, base, xmax, "joint Q")
    check_rows(d, out["k"], rk, base, xmax, "joint K")
    assert np.array_equal(h64(out["v"]), rv), "joint V: not a bit-exact copy"
    for a, p in (("k", "kp"), ("v", "vp")):
        assert np.array_equal(bits(out[a].permute(0, 2, 1, 3)), bits(out[p])), f"prefix-layout {a} differs"
    # Without the prefix-layout outputs the joint rows are the same bits.
    out2 = run_joint(d, K, Bt, ci, ts, x, kc, vc, base, pref=False)
    torch.cuda.synchronize()
    for a in ("q", "k", "v"):
        assert np.array_equal(bits(out[a]), bits(out2[a]))


FLOW_CASES = [
    # dtype, B, N, C, Lq, Lm, Ld, Hq, Hkv, D, K, Bt, per_chunk, base, splits
    (PD_BF16, 2, 4, 128, 16, 16, 24, 4, 2, 128, 2, 40, 0, 10000.0, 0),
    (PD_BF16, 1, 3, 200, 40, 8, 33, 4, 4, 64, 3, 70, 1, 0.0, 3),
    (PD_FP32, 1, 3, 64, 8, 8, 16, 4, 2, 128, 2, 9, 0, 10000.0, 2),
]


@pytest.mark.parametrize("case", FLOW_CASES, ids=[str(c) for c in FLOW_CASES])
def test_full_mask_flow(case):
    """Prefill caches -> joint rows -> dense joint attention -> decoding steps over
    the joint prefix, each against the oracle over its own joint rows."""
    dt, B, N, C, Lq, Lm, Ld, Hq, Hkv, D, K, Bt, pc, base, splits = case
    d = Dims(B, N, C, Lq, Lm, Ld, Hq, Hkv, D, dt, 0.0, pc)
    print(f"[full mask] {case}", flush=True)
    sc = 1.0 if dt == PD_BF16 else 0.25
    x = random_prefill_inputs(d, seed=C + Ld, scale=sc)
    pre = run_prefill(d, x)
    ci, ts = random_indices(d, K, Bt, seed=C)
    out = run_joint(d, K, Bt, ci, ts, x, pre["k_cache"], pre["v_cache"], base)
    Lj = K * (1 + Bt) + Lq
    dj = joint_dims(d, Lj)
    o, lse = run_dense(dj, out["q"], out["k"], out["v"], splits)
    dec = random_decode_inputs(d, seed=Ld, scale=sc)
    od, ld = run_steps(d, Lj, dec, out["kp"], out["vp"], splits)
    torch.cuda.synchronize()
    kc, vc = (h64(cache_layout(x[n])) for n in ("k_pre", "v_pre"))
    rq, rk, rv = oracle.joint_rows_ref(h64(x["q_pre"]), kc, vc, h64(x["q_qm"]), h64(x["k_qm"]), h64(x["v_qm"]),
                                       ci.cpu().numpy(), ts.cpu().numpy(), Lq, base)
    tdt = x["q_pre"].dtype
    rq, rk, rv = round_to(rq, tdt), round_to(rk, tdt), round_to(rv, tdt)
    ro, rl = oracle.joint_attention_ref(rq, rk, rv)
    assert_out_close(d, h64(o), ro, "joint attention O")
    kp, vp = rk.transpose(0, 2, 1, 3), rv.transpose(0, 2, 1, 3)
    qd, kd, vd = (h64(dec[n]) for n in ("q_dec", "k_dec", "v_dec"))
    lg, ldg = h64(lse), h64(ld)
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            assert_lse_close(d, lg[b, h], rl[b, h], rq[b, :, h], rk[b, :, g], f"joint attention (b={b}, h={h})")
            ro2, rl2 = oracle.decode_compact_unit_ref(qd, kd, vd, kp, vp, kd, vd, 0, b, h)
            assert_out_close(d, h64(od[b, :, h]), ro2, f"decode over the joint prefix (b={b}, h={h})")
            assert_lse_close(d, ldg[b, h], rl2, qd[b, :, h], np.concatenate([rk[b, :, g], kd[b, :, g]]),
                      f"decode over the joint prefix (b={b}, h={h})")


@pytest.mark.parametrize("wid", [2, 5])
def test_full_mask_full_size_sampled(wid):
    """The paper-scale workloads, in the launch configuration the benchmark times:
    sampled (sequence, head) pairs of the joint rows, the joint attention and one
    decoding step over the joint prefix."""
    w = synth.WORKLOADS[wid]
    d = w.dims()
    K, Bt, Lq = w.top_k, w.tok_budget, w.q_len
    Lj = K * (1 + Bt) + Lq
    base = 10000.0
    print(f"[full mask full size] workload {wid} {w.name} L_j={Lj}", flush=True)
    x = synth.make_prefill(w, 0, "cuda")
    kc, vc = cache_layout(x["k_pre"]), cache_layout(x["v_pre"])
    ci, ts = random_indices(d, K, Bt, seed=wid)
    out = run_joint(d, K, Bt, ci, ts, x, kc, vc, base)
    dj = joint_dims(d, Lj)
    o, lse = run_dense(dj, out["q"], out["k"], out["v"])
    dec = synth.make_decode(w, 0, 0, "cuda")
    od, ld = run_steps(d, Lj, dec, out["kp"], out["vp"])
    torch.cuda.synchronize()
    G = d.n_heads_q // d.n_heads_kv
    rng = np.random.default_rng(wid)
    pairs = [(0, 0), (d.batch - 1, d.n_heads_q - 1)] + [
        (int(rng.integers(d.batch)), int(rng.integers(d.n_heads_q))) for _ in range(2)]
    xmax = max(float(t.abs().max()) for t in x.values())
    del kc, vc
    for b, h in pairs:
        g = h // G
        chunks = ci[b].long()
        # Only the kept chunks of sequence b, head h (group g): chunk order is
        # kept, so the joint positions are those of the whole problem.
        sl = lambda t, hh: h64(t[b:b + 1].index_select(1, chunks)[:, :, :, hh:hh + 1])
        qm = lambda t, hh: h64(t[b:b + 1, 0, :, hh:hh + 1] if d.qm_per_chunk else t[b:b + 1, :, hh:hh + 1])
        local_ci = np.arange(K, dtype=np.int32)[None]
        rq, rk, rv = oracle.joint_rows_ref(
            sl(x["q_pre"], h), sl(x["k_pre"], g).transpose(0, 1, 3, 2, 4), sl(x["v_pre"], g).transpose(0, 1, 3, 2, 4),
            qm(x["q_qm"], h), qm(x["k_qm"], g), qm(x["v_qm"], g), local_ci, ts[b:b + 1].cpu().numpy(), Lq, base)
        check_rows(d, out["q"][b:b + 1, :, h:h + 1], rq, base, xmax, f"joint Q (b={b}, h={h})")
        check_rows(d, out["k"][b:b + 1, :, g:g + 1], rk, base, xmax, f"joint K (b={b}, g={g})")
        assert np.array_equal(h64(out["v"][b:b + 1, :, g:g + 1]), rv)
        assert np.array_equal(bits(out["kp"][b, g]), bits(out["k"][b, :, g]))
        tdt = x["q_pre"].dtype
        rq, rk, rv = round_to(rq, tdt), round_to(rk, tdt), round_to(rv, tdt)
        ro, rl = oracle.joint_attention_ref(rq, rk, rv)
        assert_out_close(d, h64(o[b:b + 1, :, h:h + 1]), ro, f"joint attention O (b={b}, h={h})")
        assert_lse_close(d, h64(lse[b, h]), rl[0, 0], rq[0, :, 0], rk[0, :, 0], f"joint attention (b={b}, h={h})")
        qd = h64(dec["q_dec"][b:b + 1, :, h:h + 1])
        kd, vd = (h64(dec[n][b:b + 1, :, g:g + 1]) for n in ("k_dec", "v_dec"))
        ro2, rl2 = oracle.decode_compact_unit_ref(qd, kd, vd, rk.transpose(0, 2, 1, 3), rv.transpose(0, 2, 1, 3),
                                                  kd, vd, 0, 0, 0)
        assert_out_close(d, h64(od[b, :, h]), ro2, f"decode over the joint prefix (b={b}, h={h})")
        assert_lse_close(d, h64(ld[b, h]), rl2, qd[0, :, 0], np.concatenate([rk[0, :, 0], kd[0, :, 0]]),
                  f"decode over the joint prefix (b={b}, h={h})")
