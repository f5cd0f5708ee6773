"""Benchmark of the block-sparse attention path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
prefill of every layer (chunk prefill + cache write + token/chunk summaries),
then T denoising steps, each running, for every layer, chunk scoring / top-K /
top-B selection and the sparse decode attention.

Prints one JSON line.  `value` = denoising steps per second of the whole job
(T / time of one step, prefill included); the prefill MFMA rate and the decode
attention HBM rate are reported next to it.  Inputs are resident in HBM before
the timed region starts.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA (published)
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32 vector (published; the fp32 path runs on VALU FMAs)
PEAK_HBM_GBPS = 8000.0         # MI355X HBM3E (published)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--workload", type=int, default=5, help="workload id (1-5)")
    p.add_argument("--layers", type=int, default=0, help="override the layer count (0 = workload's)")
    p.add_argument("--pool", type=int, default=2, help="distinct prefill input sets cycled over layers")
    p.add_argument("--dec-pool", type=int, default=4, help="decode input slots per layer")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="CPU time budget of the oracle sample")
    p.add_argument("--cpu-mode", choices=("auto", "sample", "full"), default="auto",
                   help="oracle timing: every unit of one job step (full; the default for workloads 1-3) or a "
                        "bounded sample extrapolated to one step (sample; the default for workloads 4-5)")
    p.add_argument("--no-workloads", action="store_true",
                   help="skip the measurements of workloads 2-4 after the timed region")
    p.add_argument("--flush-mib", type=int, default=0,
                   help="write this many MiB before every decode launch, so that each launch starts with the "
                        "last-level cache (MALL) holding none of its operands (cold numbers)")
    p.add_argument("--no-static", action="store_true",
                   help="skip the static-selection and prefill-score schedule measurements after the timed region")
    p.add_argument("--no-achievable", action="store_true",
                   help="skip the achievable-peak measurements (MFMA-rate diagnostic, device copy) after the timed region")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="before timing, copy this many MiB once (a plain copy kernel of known size for "
                        "calibrating rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    return p.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_traffic_32k_32layer_b8.md")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_10537_amd", "csrc", f)
                  for f in ("attn_bf16.hip", "pd_common.h", "pd_kernels.h", "pd_api.hip")]


def kernel_source_digest():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per decode launch from the committed rocprofv3 counter summary,
    or None when the kernel source changed since the counters were taken."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    vals = dict(l.split(":", 1) for l in text.splitlines()
                if l.startswith(("kernel_source_sha256:", "traffic_bytes_per_launch:")))
    if vals.get("kernel_source_sha256", "").strip() != kernel_source_digest():
        return None
    return int(float(vals["traffic_bytes_per_launch"]))


def algorithmic(w, layers):
    """Algorithmic FLOPs / bytes per launch of the prefill and decode attention kernels."""
    B, N, C, Lq, Lm, Ld = w.batch, w.n_chunks, w.chunk_len, w.q_len, w.m_len, w.dec_len
    Hq, Hkv, d, K, Bt = w.n_heads_q, w.n_heads_kv, w.head_dim, w.top_k, w.tok_budget
    eb = 2 if w.dtype == 0 else 4   # bytes per element: bf16 (PD_BF16 = 0) or fp32
    Sc = 1 + C + Lq + Lm
    L_kv = K * (1 + Bt) + Lq + Ld
    pre_flop = 4.0 * Sc * Sc * d * Hq * B * N
    # Reads Q, K, V of every chunk sequence once, writes O and the cache once.
    pre_bytes = eb * d * B * (N * (1 + C) * (Hq + 2 * Hkv) + (Lq + Lm) * (Hq + 2 * Hkv)
                              + N * Sc * Hq + 2 * N * (1 + C) * Hkv)
    dec_flop = 4.0 * Ld * L_kv * d * Hq * B
    # Gathered + static + own K and V rows per (b, kv head), Q read and O write per (b, q head).
    dec_bytes = eb * d * B * (2 * L_kv * Hkv + 2 * Ld * Hq)
    return pre_flop, pre_bytes, dec_flop, dec_bytes


# ---- CPU baseline: the fp64 oracle on the host cores ---------------------------------------------
# A process pool over independent units, one BLAS thread per worker: prefill units (sequence, chunk,
# query head), selection units (step, sequence) and decode units (step, sequence, query head).  Workers
# draw the workload's inputs themselves (the same seeded generator the GPU run uses) and never touch
# the GPU.  Workloads 1-3 are timed in full (every unit of one job step); workloads 4-5 are timed on a
# bounded sample of each unit kind with every worker busy, and the step time is extrapolated from the
# measured pool throughput and the unit counts.
CPU_SHARE = 16   # host cores one GPU's share of the box provides


def _cpu_host_info(workers):
    import platform
    import numpy as np
    from threadpoolctl import threadpool_info
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as f:
            model = next((l.split(":", 1)[1].strip() for l in f if l.startswith("model name")), model)
    except OSError:
        pass
    blas = [f"{i.get('internal_api')} {i.get('version')}" for i in threadpool_info() if i.get("user_api") == "blas"]
    return {"cores": workers, "affinity_cpus": len(os.sched_getaffinity(0)), "os_cpu_count": os.cpu_count(),
            "cpu_model": model, "numpy": np.__version__, "blas": ", ".join(blas) or "none found",
            "blas_threads_per_worker": 1}


_CW = {}   # per-worker state: workload, its prefill inputs (fp32 copies of the exact values), decode cache


def _cpu_worker_init(wid, full):
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)
    from paper_2606_10537_amd import synth
    w = synth.WORKLOADS[wid]
    if not full:   # one sequence, one chunk of the workload's shapes
        w = synth.Workload(**{**w.__dict__, "batch": 1, "n_chunks": 1})
    x = synth.make_prefill(w, 0, "cpu")
    _CW.update(w=w, x={k: v.float().numpy() for k, v in x.items()}, dec_t=None)


def _cpu_decode_inputs(t):
    from paper_2606_10537_amd import synth
    if _CW["dec_t"] != t:
        d = synth.make_decode(_CW["w"], 0, t, "cpu")
        _CW.update(dec={k: v.float().numpy() for k, v in d.items()}, dec_t=t)
    return _CW["dec"]


def _cpu_prefill_unit(b, n, h):
    """One prefill unit; returns (seconds, this head's Eq. 5 term, b, n)."""
    import oracle
    x, w = _CW["x"], _CW["w"]
    t0 = time.perf_counter()
    u = oracle.prefill_unit_ref(x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"], b, n, h,
                                w.q_len)
    return time.perf_counter() - t0, u["e_head"], b, n


def _cpu_select_unit(t, key_mean, tok_score):
    """Selection of step t for every sequence; returns (seconds, chunk_idx, tok_slot)."""
    import oracle
    w = _CW["w"]
    q = _cpu_decode_inputs(t)["q_dec"]
    t0 = time.perf_counter()
    ci, ts, _ = oracle.score_select_ref(q, key_mean, tok_score, w.top_k, w.tok_budget)
    return time.perf_counter() - t0, ci, ts


def _cpu_decode_unit(t, b, h, chunk_idx, tok_slot):
    """One decode unit (step t, sequence b, query head h) over the chunk cache, a transposed view of the
    worker's prefill inputs; chunk_idx (B, K) and tok_slot (B, K, B_tok) as the selection wrote them.
    Returns seconds."""
    import numpy as np
    import oracle
    x, w = _CW["x"], _CW["w"]
    dec = _cpu_decode_inputs(t)
    kc = np.transpose(x["k_pre"], (0, 1, 3, 2, 4))
    vc = np.transpose(x["v_pre"], (0, 1, 3, 2, 4))
    t0 = time.perf_counter()
    oracle.decode_unit_ref(dec["q_dec"], dec["k_dec"], dec["v_dec"], kc, vc, chunk_idx, tok_slot, x["k_qm"],
                           x["v_qm"], w.q_len, b, h)
    return time.perf_counter() - t0


def _cpu_decode_unit_sample(t, h):
    """A decode unit of the sample mode: the K kept chunks are K copies of the one chunk, the kept slots
    the first B_tok (the work does not depend on which rows are kept)."""
    import numpy as np
    w = _CW["w"]
    ci = np.zeros((1, w.top_k), dtype=np.int32)
    ts = np.tile(np.arange(1, w.tok_budget + 1, dtype=np.int32), (1, w.top_k, 1))
    return _cpu_decode_unit(t, 0, h, ci, ts)


def _cpu_select_unit_sample(t):
    import numpy as np
    w = _CW["w"]
    rng = np.random.default_rng(t)
    km = rng.standard_normal((1, max(w.top_k, 1), w.n_heads_kv, w.head_dim))
    ts = rng.standard_normal((1, km.shape[1], w.chunk_len))
    return _cpu_select_unit(t, km, ts)[0]


def cpu_baseline(w, budget_s, mode):
    """The fp64 oracle, timed on the host cores (see the section comment); returns the cpu_baseline
    object of the JSON line."""
    import concurrent.futures as cf
    import multiprocessing as mp
    import numpy as np
    workers = max(1, min(len(os.sched_getaffinity(0)), CPU_SHARE))
    for var in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[var] = "1"   # inherited by the spawned workers before they import numpy
    full = mode == "full" or (mode == "auto" and w.cid <= 3)
    B, N, C, Hq, Hkv, d, K = w.batch, w.n_chunks, w.chunk_len, w.n_heads_q, w.n_heads_kv, w.head_dim, w.top_k
    L, T = w.layers, w.steps
    info = _cpu_host_info(workers)
    ctx = mp.get_context("spawn")
    with cf.ProcessPoolExecutor(workers, mp_context=ctx, initializer=_cpu_worker_init,
                                initargs=(w.cid, full)) as ex:
        list(ex.map(time.sleep, [0.01] * workers))   # all workers up (imports, inputs) before timing
        if full:
            from paper_2606_10537_amd import synth
            x = {k: v.float().numpy() for k, v in synth.make_prefill(w, 0, "cpu").items()}
            t0 = time.perf_counter()
            futs = [ex.submit(_cpu_prefill_unit, b, n, h) for b in range(B) for n in range(N) for h in range(Hq)]
            e = np.zeros((B, N, C))
            for f in futs:
                _, eh, b, n = f.result()
                e[b, n] += eh
            import oracle
            km = oracle.key_mean_ref(x["k_pre"])
            t_pre = time.perf_counter() - t0
            for t in range(T):
                _, ci, ts = ex.submit(_cpu_select_unit, t, km, e).result()
                dfuts = [ex.submit(_cpu_decode_unit, t, b, h, ci, ts) for b in range(B) for h in range(Hq)]
                for f in dfuts:
                    f.result()
            step_s = (time.perf_counter() - t0) * L
            return {"value": T / step_s, "unit": "denoising steps/s", "kind": "oracle", "mode": "full",
                    "seconds_per_step": step_s, "prefill_s": t_pre * L, **info,
                    "sample": (f"fp64 oracle, every unit of one job step: {B * N * Hq * L} prefill units "
                               f"(S_c={1 + C + w.q_len + w.m_len}), {T * L} selections, {B * Hq * T * L} decode "
                               f"units (L_kv={K * (1 + w.tok_budget) + w.q_len + w.dec_len}), {workers} worker "
                               f"processes, 1 BLAS thread each")}

        def pool_rate(fn, args_list, share):
            """Units per second with every worker busy, on rounds of `workers` units within the budget."""
            n, t0 = 0, time.perf_counter()
            while True:
                list(ex.map(fn, *zip(*args_list)))
                n += len(args_list)
                if time.perf_counter() - t0 >= share * budget_s:
                    return n / (time.perf_counter() - t0), n

        r_pre, n_pre = pool_rate(_cpu_prefill_unit, [(0, 0, h % Hq) for h in range(workers)], 0.5)
        r_sel, n_sel = pool_rate(_cpu_select_unit_sample, [(t,) for t in range(workers)], 0.1)
        r_dec, n_dec = pool_rate(_cpu_decode_unit_sample, [(t % 4, h % Hq) for t, h in
                                                           zip(range(workers), range(workers))], 0.4)
    # one selection unit of the sample covers one sequence: B of them per (step, layer)
    units_pre, units_sel, units_dec = B * N * Hq * L, B * T * L, B * Hq * T * L
    step_s = units_pre / r_pre + units_sel / r_sel + units_dec / r_dec
    return {"value": T / step_s, "unit": "denoising steps/s", "kind": "oracle", "mode": "extrapolated",
            "seconds_per_step_extrapolated": step_s,
            "pool_units_per_s": {"prefill": r_pre, "select": r_sel, "decode": r_dec}, **info,
            "sample": (f"fp64 oracle on {workers} worker processes (1 BLAS thread each): {n_pre} prefill units "
                       f"(1 chunk x 1 head, S_c={1 + C + w.q_len + w.m_len}), {n_sel} selections (1 sequence), "
                       f"{n_dec} decode units (1 sequence x 1 head, L_kv={K * (1 + w.tok_budget) + w.q_len + w.dec_len}); "
                       f"pool throughput x unit counts of one job step ({units_pre} prefill, {units_sel} "
                       f"selection, {units_dec} decode units); extrapolated")}


def static_mode(torch, _lib, w, d, pool, dec_pool, k_cache, v_cache, key_mean, tok_rank, stream, dec_flop,
                pre_ms_layer, n_static):
    """Static-selection mode on the same caches, measured after the timed region: per layer one
    selection from the pseudo-label rows and one gather of the kept rows into a compact buffer, then
    the T-step loop of compact decodes (HIP events around every decode launch)."""
    dev = "cuda"
    L, T, K, Bt = w.layers, w.steps, w.top_k, w.tok_budget
    B, Hkv, D = w.batch, w.n_heads_kv, w.head_dim
    n_sel = K * (1 + Bt)
    sh = stream.cuda_stream
    ws_sel = torch.zeros(_lib.pd_workspace_bytes(d, K, Bt, 0, 1), dtype=torch.uint8, device=dev)
    ws_dec = torch.empty(max(16, _lib.pd_compact_workspace_bytes(d, n_sel, 0)), dtype=torch.uint8, device=dev)
    ci = torch.empty((B, K), dtype=torch.int32, device=dev)
    ts = torch.empty((B, K, Bt), dtype=torch.int32, device=dev)
    k_sel = [torch.empty((B, Hkv, n_sel, D), dtype=w.torch_dtype, device=dev) for _ in range(L)]
    v_sel = [torch.empty_like(k_sel[0]) for _ in range(L)]
    o_dec = torch.empty((B, w.dec_len, w.n_heads_q, D), dtype=w.torch_dtype, device=dev)
    dec_slots = len(dec_pool[0])

    def select_gather():
        for l in range(L):
            _lib.pd_score_select_static(d, K, Bt, pool[l % len(pool)]["q_qm"], key_mean[l], tok_rank[l], ci, ts,
                                        None, ws_sel, sh)
            _lib.pd_gather_selected(d, K, Bt, k_cache[l], v_cache[l], ci, ts, k_sel[l], v_sel[l], sh)

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(L * T)]

    def loop(record):
        i = 0
        for t in range(T):
            for l in range(L):
                dd = dec_pool[l][t % dec_slots]
                if record:
                    ev[i][0].record(stream)
                _lib.pd_sparse_decode_attn_compact(d, n_sel, dd["q_dec"], dd["k_dec"], dd["v_dec"], k_sel[l],
                                                   v_sel[l], pool[l % len(pool)]["k_qm"],
                                                   pool[l % len(pool)]["v_qm"], n_static, o_dec, None, 0, ws_dec, sh)
                if record:
                    ev[i][1].record(stream)
                i += 1

    select_gather()
    loop(False)
    torch.cuda.synchronize()
    s0, s1, s2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    s0.record(stream)
    select_gather()
    s1.record(stream)
    loop(True)
    s2.record(stream)
    torch.cuda.synchronize()
    sg_ms = s0.elapsed_time(s1)
    loop_ms = s1.elapsed_time(s2)
    launch_ms = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    return {"steps_per_s": round(T / (loop_ms * 1e-3), 3),
            "job_steps_per_s": round(T / ((pre_ms_layer * L + sg_ms + loop_ms) * 1e-3), 3),
            "loop_ms": round(loop_ms, 3),
            "select_gather_ms_per_layer": round(sg_ms / L, 4),
            "decode_launch_ms": round(launch_ms, 5),
            "decode_tflops": round(dec_flop / (launch_ms * 1e-3) / 1e12, 2),
            "note": "selection once per layer from the pseudo-label rows, kept rows compacted once; decode over "
                    "the compact buffer; same caches, decode inputs and flop count as the per-step mode"}


def prefill_score_mode(torch, _lib, w, d, pool, prefill_bufs, k_cache, v_cache, tok_rank, key_mean, stream,
                       static_loop_ms):
    """The paper's own schedule with the prefill-time chunk score, measured after the timed region:
    every layer's prefill also writes the chunk scores, the K lowest chunks are kept and their kept
    rows compacted once; the T-step loop of compact decodes is the one static_mode timed (same kernels,
    sizes and decode inputs; decode time does not depend on which rows were kept)."""
    dev = "cuda"
    L, T, K, Bt = w.layers, w.steps, w.top_k, w.tok_budget
    B, Hkv, D = w.batch, w.n_heads_kv, w.head_dim
    n_sel = K * (1 + Bt)
    sh = stream.cuda_stream
    o_pre, tok_score, ws_pre = prefill_bufs
    cs = torch.empty((B, w.n_chunks), dtype=torch.float32, device=dev)
    ci = torch.empty((B, K), dtype=torch.int32, device=dev)
    ts = torch.empty((B, K, Bt), dtype=torch.int32, device=dev)
    k_sel = torch.empty((B, Hkv, n_sel, D), dtype=w.torch_dtype, device=dev)
    v_sel = torch.empty_like(k_sel)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(L)]

    def run(record):
        for l in range(L):
            x = pool[l % len(pool)]
            if record:
                ev[l][0].record(stream)
            _lib.pd_prefill_chunks(d, x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"], o_pre,
                                   k_cache[l], v_cache[l], tok_score, tok_rank[l], key_mean[l], ws_pre, sh,
                                   chunk_score=cs)
            if record:
                ev[l][1].record(stream)
            _lib.pd_select_ranked(d, K, Bt, cs, 1, tok_rank[l], ci, ts, sh)
            _lib.pd_gather_selected(d, K, Bt, k_cache[l], v_cache[l], ci, ts, k_sel, v_sel, sh)
            if record:
                ev[l][2].record(stream)

    run(False)
    torch.cuda.synchronize()
    run(True)
    torch.cuda.synchronize()
    pre = sum(a.elapsed_time(b) for a, b, _ in ev) / L
    sel = sum(b.elapsed_time(c) for _, b, c in ev) / L
    return {"prefill_ms_per_layer": round(pre, 3),
            "select_gather_ms_per_layer": round(sel, 4),
            "job_steps_per_s": round(T / (((pre + sel) * L + static_loop_ms) * 1e-3), 3),
            "note": "prefill also writes the chunk scores (attention mass of the query and pseudo-label rows on "
                    "each chunk's content); the K lowest kept once per layer, kept rows compacted; decode loop "
                    "as in static_mode"}


def full_mask_mode(torch, _lib, w, d, pool, dec_pool, prefill_bufs, k_cache, v_cache, tok_rank, key_mean, stream,
                   rope_base=500000.0):
    """Full-mask cache construction, measured after the timed region: per layer the prefill with the
    chunk score, the K lowest chunks kept, their kept rows and the query rows moved to continuous
    positions (rotary re-rotation) and attended densely together; then the T-step loop of compact
    decodes whose prefix is the L_j joint rows (same row count as the static mode's prefix + static
    rows, so the same decode flop count)."""
    from paper_2606_10537_amd import synth
    dev = "cuda"
    L, T, K, Bt = w.layers, w.steps, w.top_k, w.tok_budget
    B, Hq, Hkv, D = w.batch, w.n_heads_q, w.n_heads_kv, w.head_dim
    Lj = K * (1 + Bt) + w.q_len
    dj = synth.Workload(**{**w.__dict__, "dec_len": Lj}).dims()
    sh = stream.cuda_stream
    o_pre, tok_score, ws_pre = prefill_bufs
    dt = w.torch_dtype
    cs = torch.empty((B, w.n_chunks), dtype=torch.float32, device=dev)
    ci = torch.empty((B, K), dtype=torch.int32, device=dev)
    ts = torch.empty((B, K, Bt), dtype=torch.int32, device=dev)
    qj = torch.empty((B, Lj, Hq, D), dtype=dt, device=dev)
    kj, vj = torch.empty((B, Lj, Hkv, D), dtype=dt, device=dev), torch.empty((B, Lj, Hkv, D), dtype=dt, device=dev)
    oj = torch.empty_like(qj)
    kp = [torch.empty((B, Hkv, Lj, D), dtype=dt, device=dev) for _ in range(L)]
    vp = [torch.empty_like(kp[0]) for _ in range(L)]
    ws_joint = torch.empty(max(16, _lib.pd_compact_workspace_bytes(dj, 0, 0)), dtype=torch.uint8, device=dev)
    ws_dec = torch.empty(max(16, _lib.pd_compact_workspace_bytes(d, Lj, 0)), dtype=torch.uint8, device=dev)
    o_dec = torch.empty((B, w.dec_len, Hq, D), dtype=dt, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(L)]
    dec_slots = len(dec_pool[0])

    def build(record):
        for l in range(L):
            x = pool[l % len(pool)]
            if record:
                ev[l][0].record(stream)
            _lib.pd_prefill_chunks(d, x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"], o_pre,
                                   k_cache[l], v_cache[l], tok_score, tok_rank[l], key_mean[l], ws_pre, sh,
                                   chunk_score=cs)
            if record:
                ev[l][1].record(stream)
            _lib.pd_select_ranked(d, K, Bt, cs, 1, tok_rank[l], ci, ts, sh)
            if record:
                ev[l][2].record(stream)
            _lib.pd_gather_joint(d, K, Bt, ci, ts, x["q_pre"], k_cache[l], v_cache[l], x["q_qm"], x["k_qm"],
                                 x["v_qm"], rope_base, qj, kj, vj, kp[l], vp[l], sh)
            if record:
                ev[l][3].record(stream)
            _lib.pd_sparse_decode_attn_compact(dj, 0, qj, kj, vj, None, None, None, None, 0, oj, None, 0,
                                               ws_joint, sh)
            if record:
                ev[l][4].record(stream)

    def loop():
        for t in range(T):
            for l in range(L):
                dd = dec_pool[l][t % dec_slots]
                _lib.pd_sparse_decode_attn_compact(d, Lj, dd["q_dec"], dd["k_dec"], dd["v_dec"], kp[l], vp[l], None,
                                                   None, 0, o_dec, None, 0, ws_dec, sh)

    build(False)
    loop()
    torch.cuda.synchronize()
    build(True)
    s1, s2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s1.record(stream)
    loop()
    s2.record(stream)
    torch.cuda.synchronize()
    per = [sum(e[i].elapsed_time(e[i + 1]) for e in ev) / L for i in range(4)]
    loop_ms = s1.elapsed_time(s2)
    joint_flop = 4.0 * B * Hq * Lj * Lj * D
    return {"prefill_ms_per_layer": round(per[0], 3),
            "select_ms_per_layer": round(per[1], 4),
            "gather_joint_ms_per_layer": round(per[2], 4),
            "joint_attn_ms_per_layer": round(per[3], 4),
            "joint_attn_tflops": round(joint_flop / (per[3] * 1e-3) / 1e12, 2),
            "loop_ms": round(loop_ms, 3),
            "job_steps_per_s": round(T / ((sum(per) * L + loop_ms) * 1e-3), 3),
            "joint_rows": Lj, "rope_base": rope_base,
            "note": "prefill with the chunk score; K lowest kept; kept rows + query rows re-rotated to continuous "
                    "positions and attended densely together (the one-layer slice of the joint re-encoding); "
                    "decode loop over the L_j joint rows"}


def achievable_peaks(torch, dev):
    """Achievable (not published) peaks on this GPU, measured after the timed region: the library's
    MFMA-rate diagnostic (register-only v_mfma_f32_32x32x16_bf16 chains on every CU) and a
    device-to-device copy of 4 GiB (read + write bytes)."""
    from paper_2606_10537_amd import _lib
    n_wg, iters = 2048, 4000
    sink = torch.empty(n_wg * 256, dtype=torch.float32, device=dev)
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    _lib.pd_mfma_rate_probe(n_wg, iters, sink)
    s.record()
    for _ in range(3):
        _lib.pd_mfma_rate_probe(n_wg, iters, sink)
    e.record()
    torch.cuda.synchronize()
    mfma = 3.0 * n_wg * 4 * iters * 8 * 32768 / (s.elapsed_time(e) * 1e-3) / 1e12
    src = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    s.record()
    for _ in range(5):
        dst.copy_(src)
    e.record()
    torch.cuda.synchronize()
    copy = 2.0 * src.numel() * 5 / (s.elapsed_time(e) * 1e-3) / 1e9
    del src, dst
    return {"mfma_tflops": round(mfma, 1), "hbm_gbps": round(copy, 1),
            "method": "pd_mfma_rate_probe (2048 workgroups x 4 waves x 4 independent 32x32x16 bf16 chains) "
                      "and a 4 GiB device copy (read + write bytes)"}


def measure(torch, _lib, w, steps, warmup, pool_n=2, dec_pool_n=4, flush_mib=0, calib_copy_mib=0, log=""):
    """Inputs resident in HBM, then `warmup` untimed and `steps` timed job steps of workload w: prefill of
    every layer, then T denoising steps of (selection, sparse decode) for every layer.  HIP events on the
    launch stream around every prefill, selection and decode launch.  Returns the timings and the
    resident buffers (the select-once schedules reuse them)."""
    from paper_2606_10537_amd import synth
    d = w.dims()
    dev = "cuda"
    dt = w.torch_dtype
    B, N, C, Hq, Hkv, D = w.batch, w.n_chunks, w.chunk_len, w.n_heads_q, w.n_heads_kv, w.head_dim
    L, T, K, Bt, Ld = w.layers, w.steps, w.top_k, w.tok_budget, w.dec_len
    n_static = w.q_len

    pool = [synth.make_prefill(w, layer=i, device=dev) for i in range(min(pool_n, L))]
    dec_slots = max(1, dec_pool_n)
    dec_pool = [[synth.make_decode(w, layer=l, step=s, device=dev) for s in range(dec_slots)] for l in range(L)]
    o_pre = torch.empty((B, N, d.seq_len, Hq, D), dtype=dt, device=dev)
    k_cache = [torch.empty((B, N, Hkv, C + 1, D), dtype=dt, device=dev) for _ in range(L)]
    v_cache = [torch.empty((B, N, Hkv, C + 1, D), dtype=dt, device=dev) for _ in range(L)]
    tok_score = torch.empty((B, N, C), dtype=torch.float32, device=dev)
    tok_rank = [torch.empty((B, N, C), dtype=torch.int32, device=dev) for _ in range(L)]
    key_mean = [torch.empty((B, N, Hkv, D), dtype=torch.float32, device=dev) for _ in range(L)]
    ws_pre = torch.empty(_lib.pd_workspace_bytes(d, which=0), dtype=torch.uint8, device=dev)
    ws_sel = torch.zeros(_lib.pd_workspace_bytes(d, K, Bt, 0, 1), dtype=torch.uint8, device=dev)
    ws_dec = torch.empty(max(16, _lib.pd_workspace_bytes(d, K, Bt, 0, 2)), dtype=torch.uint8, device=dev)
    chunk_idx = torch.empty((B, K), dtype=torch.int32, device=dev)
    tok_slot = torch.empty((B, K, Bt), dtype=torch.int32, device=dev)
    o_dec = torch.empty((B, Ld, Hq, D), dtype=dt, device=dev)
    splits = _lib.pd_decode_splits(d, K, Bt, n_static, 0)
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream

    flush = torch.empty(flush_mib << 20, dtype=torch.uint8, device=dev) if flush_mib else None
    E = lambda: torch.cuda.Event(enable_timing=True)
    ev_pre = [(E(), E()) for _ in range(L)]
    ev_dec = [(E(), E()) for _ in range(L * T)]
    ev_mid = E()

    def one_step(record):
        for l in range(L):
            x = pool[l % len(pool)]
            if record:
                ev_pre[l][0].record(stream)
            _lib.pd_prefill_chunks(d, x["q_pre"], x["k_pre"], x["v_pre"], x["q_qm"], x["k_qm"], x["v_qm"], o_pre,
                                   k_cache[l], v_cache[l], tok_score, tok_rank[l], key_mean[l], ws_pre, sh)
            if record:
                ev_pre[l][1].record(stream)
        if record:
            ev_mid.record(stream)
        i = 0
        for t in range(T):
            for l in range(L):
                dd = dec_pool[l][t % dec_slots]
                _lib.pd_score_select(d, K, Bt, dd["q_dec"], key_mean[l], tok_rank[l], chunk_idx, tok_slot, None,
                                     ws_sel, sh)
                if flush is not None:
                    flush.fill_(t & 0xFF)
                if record:
                    ev_dec[i][0].record(stream)
                _lib.pd_sparse_decode_attn(d, K, Bt, dd["q_dec"], dd["k_dec"], dd["v_dec"], k_cache[l], v_cache[l],
                                           chunk_idx, tok_slot, pool[l % len(pool)]["k_qm"],
                                           pool[l % len(pool)]["v_qm"], n_static, o_dec, None, 0, ws_dec, sh)
                if record:
                    ev_dec[i][1].record(stream)
                i += 1

    if calib_copy_mib:
        src = torch.empty(calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(warmup):
        one_step(False)
    torch.cuda.synchronize()

    pre_ms, dec_ms, dec_kernel_ms, sel_ms, step_ms = [], [], [], [], []
    start, end = E(), E()
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    for s in range(steps):
        start.record(stream)
        one_step(True)
        end.record(stream)
        torch.cuda.synchronize()
        step_ms.append(start.elapsed_time(end))
        pre_ms.append(start.elapsed_time(ev_mid))
        dec_ms.append(ev_mid.elapsed_time(end))
        dec_kernel_ms.extend(a.elapsed_time(b) for a, b in ev_dec)
        # between two decode launches: the next selection's launches and the gaps around them
        sel_ms.extend(ev_dec[i - 1][1].elapsed_time(ev_dec[i][0]) for i in range(1, len(ev_dec)))
        print(f"[bench]{log} step {s}: {step_ms[-1]:.1f} ms (prefill {pre_ms[-1]:.1f} ms, decode loop "
              f"{dec_ms[-1]:.1f} ms)", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    return {"d": d, "ms": sum(step_ms) / len(step_ms), "pre_ms_layer": sum(pre_ms) / len(pre_ms) / L,
            "dec_loop_ms": sum(dec_ms) / len(dec_ms), "dec_kern_ms": sum(dec_kernel_ms) / len(dec_kernel_ms),
            "sel_ms": sum(sel_ms) / len(sel_ms) if sel_ms else 0.0, "splits": splits, "wall": wall,
            "bufs": {"pool": pool, "dec_pool": dec_pool, "o_pre": o_pre, "k_cache": k_cache, "v_cache": v_cache,
                     "tok_score": tok_score, "tok_rank": tok_rank, "key_mean": key_mean, "ws_pre": ws_pre,
                     "stream": stream}}


def rates(w, m):
    """Throughput and roofline figures of one measure() result."""
    bf16 = w.dtype == 0
    L, T = w.layers, w.steps
    pre_flop, pre_bytes, dec_flop, dec_bytes = algorithmic(w, L)
    peak_c = PEAK_BF16_TFLOPS if bf16 else PEAK_FP32_TFLOPS
    dk = m["dec_kern_ms"] * 1e-3
    dec_tflops, dec_gbps = dec_flop / dk / 1e12, dec_bytes / dk / 1e9
    ridge = peak_c * 1e12 / (PEAK_HBM_GBPS * 1e9)
    bound = ("mfma" if bf16 else "alu") if dec_flop / dec_bytes > ridge else "hbm"
    binding = max(dec_flop / (peak_c * 1e12), dec_bytes / (PEAK_HBM_GBPS * 1e9)) / dk
    pre_tflops = pre_flop / (m["pre_ms_layer"] * 1e-3) / 1e12
    return {"dec_flop": dec_flop, "dec_bytes": dec_bytes, "dec_tflops": dec_tflops, "dec_gbps": dec_gbps,
            "peak_c": peak_c, "bound": bound, "binding_frac": binding, "pre_tflops": pre_tflops,
            "job_steps_per_s": T / (m["ms"] * 1e-3), "decode_steps_per_s": T / (m["dec_loop_ms"] * 1e-3)}


# Every input tensor is drawn from its own torch.Generator (synth.seed_of).
SEED_RULE = "({base}) * 1000003 + crc32('workload/layer/tensor/step')"


def workload_summary(w, m):
    """The per-workload object of the JSON line."""
    r = rates(w, m)
    unit = "GB/s" if r["bound"] == "hbm" else "TFLOP/s"
    achieved = r["dec_gbps"] if r["bound"] == "hbm" else r["dec_tflops"]
    peak = PEAK_HBM_GBPS if r["bound"] == "hbm" else r["peak_c"]
    ctx = f"{w.context // 1024}K" if w.context >= 1024 else f"{w.context}-token"
    return {"workload": f"{ctx} context ({w.name}): B={w.batch}, layers={w.layers}, N={w.n_chunks}, "
                        f"C={w.chunk_len}, L_q={w.q_len}, L_m={w.m_len}, L_d={w.dec_len}, "
                        f"H_q/H_kv={w.n_heads_q}/{w.n_heads_kv}, d={w.head_dim}, K={w.top_k}, "
                        f"B_tok={w.tok_budget}, T={w.steps}",
            "job_steps_per_s": round(r["job_steps_per_s"], 3), "ms_per_step": round(m["ms"], 4),
            "decode_steps_per_s": round(r["decode_steps_per_s"], 3),
            "decode_us_per_launch": round(m["dec_kern_ms"] * 1e3, 2),
            "select_and_gaps_us_per_step": round(m["sel_ms"] * 1e3, 2),
            "decode_splits": m["splits"],
            "decode_roofline": {"bound": r["bound"], "achieved": round(achieved, 2), "peak": peak, "unit": unit,
                                "frac": round(achieved / peak, 4)},
            "decode_tflops": round(r["dec_tflops"], 2), "decode_algorithmic_gbps": round(r["dec_gbps"], 1),
            "decode_binding_roof_frac": round(r["binding_frac"], 4),
            "prefill_ms_per_layer": round(m["pre_ms_layer"], 4), "prefill_tflops": round(r["pre_tflops"], 2),
            "prefill_mfma_frac": round(r["pre_tflops"] / r["peak_c"], 4)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path shards by "
              "sequence with no communication, so multi-GPU figures are not produced.", file=sys.stderr)
        sys.exit(2)
    from paper_2606_10537_amd import synth
    w = synth.WORKLOADS[args.workload]
    if args.layers:
        w = synth.Workload(**{**w.__dict__, "layers": args.layers})
    cpu = None
    if not args.no_cpu_baseline:
        # Before any GPU work: the oracle's worker processes start from a process that has not
        # initialised the GPU, and nothing else runs on the host meanwhile.
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_seconds, args.cpu_mode)
    import torch

    from paper_2606_10537_amd import _lib
    _lib.load()
    m = measure(torch, _lib, w, args.steps, args.warmup, args.pool, args.dec_pool, args.flush_mib,
                args.calib_copy_mib)
    d = m["d"]
    r = rates(w, m)
    bf16 = w.dtype == _lib.PD_BF16
    B, T, L, D = w.batch, w.steps, w.layers, w.head_dim
    if r["bound"] != "hbm":
        roof = {"bound": r["bound"], "achieved": round(r["dec_tflops"], 2), "peak": r["peak_c"], "unit": "TFLOP/s",
                "frac": round(r["dec_tflops"] / r["peak_c"], 4)}
    else:
        roof = {"bound": "hbm", "achieved": round(r["dec_gbps"], 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                "frac": round(r["dec_gbps"] / PEAK_HBM_GBPS, 4)}
    kname = f"decode_{'bf16' if bf16 else 'f32'}_kernel<{D}>"
    roof.update({"kernel": f"{kname} (pd_sparse_decode_attn, one launch per layer and step)",
                 "traffic": measured_traffic() if (args.workload == 5 and not args.layers) else None,
                 "launch_ms": round(m["dec_kern_ms"], 5), "flop_per_launch": r["dec_flop"],
                 "bytes_per_launch": r["dec_bytes"]})
    traffic = roof.get("traffic")
    summ = workload_summary(w, m)
    res = {
        "metric": "denoising steps/sec + decode-attn HBM GB/s + prefill MFMA TFLOP/s at 32K",
        "value": round(r["job_steps_per_s"], 3),
        "unit": "denoising steps/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(m["ms"], 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32", "data": "synthetic",
        "config": {"workload": summ["workload"], "global_batch": B, "seq_len": w.context,
                   "parallelism": "single GPU", "decode_splits": m["splits"],
                   "seed": SEED_RULE.format(base=20260 + w.cid)},
        "decode_steps_per_s": round(r["decode_steps_per_s"], 3),
        "decode_attn_hbm_gbps": round(r["dec_gbps"], 1),
        "decode_attn_hbm_frac": round(r["dec_gbps"] / PEAK_HBM_GBPS, 4),
        "decode_attn_tflops": round(r["dec_tflops"], 2),
        "select_and_gaps_us_per_step": summ["select_and_gaps_us_per_step"],
        "prefill_ms_per_layer": round(m["pre_ms_layer"], 3),
        "prefill_tflops": round(r["pre_tflops"], 2),
        "prefill_mfma_frac": round(r["pre_tflops"] / r["peak_c"], 4),
        "compute_peak_tflops": r["peak_c"],
        "decode_dram_gbps": round(traffic / (m["dec_kern_ms"] * 1e-3) / 1e9, 1) if traffic else None,
        "decode_binding_roof_frac": round(r["binding_frac"], 4),
        "cold_flush_mib": args.flush_mib,
        "roofline": roof,
        "wall_s": round(m["wall"], 3),
    }
    bufs = m.pop("bufs")
    if not args.no_static:
        stream = bufs["stream"]
        res["static_mode"] = static_mode(torch, _lib, w, d, bufs["pool"], bufs["dec_pool"], bufs["k_cache"],
                                         bufs["v_cache"], bufs["key_mean"], bufs["tok_rank"], stream, r["dec_flop"],
                                         m["pre_ms_layer"], w.q_len)
        prefill_bufs = (bufs["o_pre"], bufs["tok_score"], bufs["ws_pre"])
        res["prefill_score_mode"] = prefill_score_mode(torch, _lib, w, d, bufs["pool"], prefill_bufs,
                                                       bufs["k_cache"], bufs["v_cache"], bufs["tok_rank"],
                                                       bufs["key_mean"], stream, res["static_mode"]["loop_ms"])
        res["full_mask_mode"] = full_mask_mode(torch, _lib, w, d, bufs["pool"], bufs["dec_pool"], prefill_bufs,
                                               bufs["k_cache"], bufs["v_cache"], bufs["tok_rank"], bufs["key_mean"],
                                               stream)
    del bufs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    if not args.no_achievable:
        ach = achievable_peaks(torch, "cuda")
        res["achievable"] = ach
        if roof["bound"] != "alu":   # the achievable rates are bf16 MFMA and HBM
            roof["frac_of_achievable"] = round(roof["achieved"] / (ach["mfma_tflops"] if roof["bound"] == "mfma"
                                                                   else ach["hbm_gbps"]), 4)
        if bf16:
            res["prefill_frac_of_achievable"] = round(r["pre_tflops"] / ach["mfma_tflops"], 4)
    if not args.no_workloads:
        # The other GPU workloads of the method's configurations, one after another after the timed
        # region (each with its own resident inputs).
        res["workloads"] = {}
        for wid in (2, 3, 4):
            if wid == args.workload:
                continue
            wk = synth.WORKLOADS[wid]
            mk = measure(torch, _lib, wk, steps=3, warmup=1, log=f" workload {wid}")
            mk.pop("bufs")
            res["workloads"][str(wid)] = workload_summary(wk, mk)
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
            if wid == 4:
                # Its per-step working set (143 MB) fits the 256 MB MALL: the decode once more with
                # a 512 MiB write between the selection and each decode launch, MALL cold.
                mk = measure(torch, _lib, wk, steps=1, warmup=1, flush_mib=512, log=f" workload {wid}, MALL cold")
                mk.pop("bufs")
                res["workloads"][str(wid)]["decode_us_per_launch_mall_cold"] = round(mk["dec_kern_ms"] * 1e3, 2)
                res["workloads"][str(wid)]["mall_cold_flush_mib"] = 512
                torch.cuda.synchronize()
                torch.cuda.empty_cache()
    if cpu is not None:
        res["cpu_baseline"] = cpu
    print(json.dumps(res))


if __name__ == "__main__":
    main()
