"""C-ABI boundary tests that run without a GPU.

The library must load, export every symbol include/pd.h declares, and reject
bad arguments on the host before anything is launched (so these calls never
reach the HIP runtime).  Pointers here are fake, aligned or misaligned
integers: validation only inspects them.
"""

import ctypes
import os
import re

import pytest

from paper_2606_10537_amd import _lib
from paper_2606_10537_amd._lib import PD_BF16, PD_FP32, Dims, PdError

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
A = 1 << 20          # a fake, 16-byte aligned address
MIS = A + 8          # misaligned


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def header_symbols():
    with open(os.path.join(ROOT, "include", "pd.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(pd_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    syms = header_symbols()
    assert set(syms) == set(_lib.EXPORTS)
    for s in syms:
        assert hasattr(lib, s), s


def test_version_and_status_strings(lib):
    assert b"gfx950" in lib.pd_version()
    for code, name in _lib.STATUS.items():
        assert lib.pd_status_string(code).decode() == name


def dims(**kw):
    base = dict(batch=1, n_chunks=4, chunk_len=128, q_len=16, m_len=32, dec_len=32, n_heads_q=4,
                n_heads_kv=4, head_dim=64, dtype=PD_BF16)
    base.update(kw)
    return Dims(**base)


def prefill(d, ws=A, wsn=1 << 30, **ptrs):
    names = ["q_pre", "k_pre", "v_pre", "q_qm", "k_qm", "v_qm", "o", "k_cache", "v_cache", "tok_score", "tok_rank",
             "key_mean", "chunk_score"]
    args = [ptrs.get(n, A) for n in names]
    lib = _lib.load()
    dd = d.c() if d is not None else None
    return lib.pd_prefill_chunks(ctypes.byref(dd) if dd is not None else None, *args, ws, wsn, None)


def test_prefill_validation(lib):
    assert prefill(None) == 1
    assert prefill(dims(batch=0)) == 2
    assert prefill(dims(n_chunks=1025)) == 2
    assert prefill(dims(chunk_len=0)) == 2
    assert prefill(dims(chunk_len=5000)) == 2
    assert prefill(dims(q_len=0)) == 2
    assert prefill(dims(m_len=-1)) == 2
    assert prefill(dims(qm_per_chunk=2)) == 2
    assert prefill(dims(n_heads_q=6, n_heads_kv=4)) == 3
    assert prefill(dims(head_dim=96)) == 3
    assert prefill(dims(dtype=7)) == 3
    assert prefill(dims(), q_pre=None) == 1
    assert b"q_pre" in lib.pd_last_error_message()
    assert prefill(dims(), key_mean=None) == 1
    assert prefill(dims(), tok_rank=None) == 1
    assert prefill(dims(), o=MIS) == 4
    assert prefill(dims(), ws=None) == 5
    assert prefill(dims(), wsn=16) == 5
    assert prefill(dims(), ws=MIS) == 4
    assert prefill(dims(tok_score_dir=2)) == 2
    assert prefill(dims(), chunk_score=MIS) == 4


def test_select_validation(lib):
    d = dims()
    c = ctypes.byref(d.c())
    ws = _lib.pd_workspace_bytes(d, 2, 64, 0, 1)
    assert ws > 0
    call = lambda k, bt, q=A, cs=None, w=A, wn=ws: lib.pd_score_select(c, k, bt, q, A, A, A, A, cs, w, wn, None)
    assert call(0, 64) == 2
    assert call(5, 64) == 2          # top_k > N
    assert call(2, 0) == 2
    assert call(2, 129) == 2         # tok_budget > C
    assert call(2, 64, q=None) == 1
    assert call(2, 64, cs=MIS) == 4
    assert call(2, 64, wn=ws - 1) == 5


def test_decode_validation(lib):
    d = dims(dtype=PD_BF16)
    c = ctypes.byref(d.c())

    def call(k=2, bt=64, n_static=16, splits=1, ks=A, o=A, w=A, wn=1 << 30, lse=None):
        return lib.pd_sparse_decode_attn(c, k, bt, A, A, A, A, A, A, A, ks, ks, n_static, o, lse, splits, w, wn, None)

    assert call(k=0) == 2
    assert call(k=5) == 2
    assert call(bt=200) == 2
    assert call(n_static=49) == 2     # > q_len + m_len
    assert call(n_static=-1) == 2
    assert call(splits=65) == 2
    assert call(ks=None) == 1         # static rows requested but not given
    assert call(o=None) == 1
    assert call(lse=MIS) == 4
    need = _lib.pd_workspace_bytes(d, 2, 64, 4, 2)
    assert need > 0
    assert call(splits=4, wn=need - 1) == 5
    assert call(splits=4, w=None) == 5


def test_noalloc_select_validation(lib):
    """The scratch-array selection checks its arguments and rejects sizes beyond its 4 MiB array on the
    host, before it looks up the device array (so none of these calls touches the HIP runtime)."""
    d = dims()
    c = ctypes.byref(d.c())
    call = lambda k=2, bt=64, q=A, ci=A, cs=None, dd=c: lib.pd_score_select_noalloc(dd, k, bt, q, A, A, ci, A, cs,
                                                                                    None)
    assert call(dd=None) == 1
    assert call(k=0) == 2
    assert call(k=5) == 2
    assert call(bt=129) == 2
    assert call(q=None) == 1
    assert call(ci=MIS) == 4
    assert call(cs=MIS) == 4
    big = dims(batch=64, n_chunks=1024, chunk_len=64, n_heads_q=64, n_heads_kv=8, dec_len=512)
    assert 64 * 1024 * 64 * 4 * 4 > 4 << 20
    assert call(dd=ctypes.byref(big.c())) == 2
    assert b"scratch" in lib.pd_last_error_message()


def test_static_mode_validation(lib):
    d = dims()
    c = ctypes.byref(d.c())
    ws = _lib.pd_workspace_bytes(d, 2, 64, 0, 1)
    sel = lambda k=2, bt=64, q=A, wn=ws, dd=c: lib.pd_score_select_static(dd, k, bt, q, A, A, A, A, None, A, wn, None)
    assert sel(k=0) == 2
    assert sel(bt=129) == 2
    assert sel(q=None) == 1
    assert sel(wn=ws - 1) == 5
    assert sel(dd=ctypes.byref(dims(m_len=0).c())) == 2
    gat = lambda k=2, bt=64, ks=A: lib.pd_gather_selected(c, k, bt, A, A, A, A, ks, A, None)
    assert gat(k=5) == 2
    assert gat(bt=0) == 2
    assert gat(ks=None) == 1
    cmp_ = lambda n=10, ks=A, ns=16, sp=0, lse=None: lib.pd_sparse_decode_attn_compact(
        c, n, A, A, A, ks, ks, A, A, ns, A, lse, sp, A, 1 << 30, None)
    assert cmp_(n=-1) == 2
    assert cmp_(n=(1 << 20) + 1) == 2
    assert cmp_(ks=None) == 1
    assert cmp_(ns=49) == 2
    assert cmp_(sp=65) == 2
    assert cmp_(lse=MIS) == 4
    assert _lib.pd_compact_workspace_bytes(d, -1, 0) == 0
    assert _lib.pd_compact_workspace_bytes(d, 100, 1) == 0
    assert _lib.pd_compact_workspace_bytes(d, 100, 3) >= 3 * 1 * 4 * 32 * 65 * 4


def test_decode_row_offsets_bounded(lib):
    """A decode whose KV row index times H_kv * d reaches 2^31 is rejected on the host (the kernels
    address static and own rows with 32-bit element offsets), for both decode entry points and the
    size queries; nothing is launched."""
    d = dims(n_heads_q=32, n_heads_kv=32, head_dim=128, q_len=16, m_len=32, dec_len=32)
    c = ctypes.byref(d.c())
    n_sel = 1 << 20
    assert (n_sel + 16 + 32) * 32 * 128 >= 1 << 31
    st = lib.pd_sparse_decode_attn_compact(c, n_sel, A, A, A, A, A, A, A, 16, A, None, 0, A, 1 << 40, None)
    assert st == 2
    assert b"2^31" in lib.pd_last_error_message()
    assert _lib.pd_compact_workspace_bytes(d, n_sel, 0) == 0
    # the gathered entry point: K * (1 + B_tok) prefix rows over the same bound
    dg = dims(n_heads_q=32, n_heads_kv=32, head_dim=128, n_chunks=1024, chunk_len=4096, q_len=16, m_len=32,
              dec_len=32)
    assert _lib.pd_workspace_bytes(dg, 1024, 4096, 0, 2) == 0
    # one sequence's cache alone already exceeds the per-sequence bound of check_dims here
    assert lib.pd_sparse_decode_attn(ctypes.byref(dg.c()), 1024, 4096, A, A, A, A, A, A, A, A, A, 16, A, None,
                                     0, A, 1 << 40, None) == 2


def test_launch_grids_bounded(lib):
    """A call whose decode grid (work items x shards) or chunk-score grid (sequences x heads x 128-row
    splits) would not fit one launch dimension is rejected on the host, and the size queries return 0;
    nothing is launched."""
    d = dims(batch=1 << 20, n_chunks=1, chunk_len=1, q_len=1, m_len=0, dec_len=1 << 19, n_heads_q=1,
             n_heads_kv=1, head_dim=128)
    c = ctypes.byref(d.c())
    assert (1 << 20) * ((1 << 19) // 256) >= 1 << 31           # decode work items
    assert lib.pd_score_select(c, 1, 1, A, A, A, A, A, None, A, 1 << 40, None) == 2
    assert b"too large" in lib.pd_last_error_message()
    assert lib.pd_score_select_noalloc(c, 1, 1, A, A, A, A, A, None, None) == 2
    assert _lib.pd_workspace_bytes(d, 0, 0, 0, 1) == 0
    assert lib.pd_sparse_decode_attn(c, 1, 1, A, A, A, A, A, A, A, A, A, 1, A, None, 0, A, 1 << 40, None) == 2
    assert b"too large" in lib.pd_last_error_message()
    assert _lib.pd_workspace_bytes(d, 1, 1, 0, 2) == 0
    assert _lib.pd_compact_workspace_bytes(d, 2, 0) == 0
    # the same sizes at batch 1 are accepted by the size queries
    d1 = dims(batch=1, n_chunks=1, chunk_len=1, q_len=1, m_len=0, dec_len=1 << 19, n_heads_q=1, n_heads_kv=1,
              head_dim=128)
    assert _lib.pd_workspace_bytes(d1, 0, 0, 0, 1) > 0


def test_select_ranked_validation(lib):
    c = ctypes.byref(dims().c())
    call = lambda k=2, bt=64, cs=A, low=1, tr=A, ci=A, dd=c: lib.pd_select_ranked(dd, k, bt, cs, low, tr, ci, A, None)
    assert call(dd=None) == 1
    assert call(k=0) == 2
    assert call(k=5) == 2            # top_k > N
    assert call(bt=129) == 2         # tok_budget > C
    assert call(low=2) == 2
    assert call(cs=None) == 1
    assert call(tr=None) == 1
    assert call(ci=MIS) == 4
    assert call(dd=ctypes.byref(dims(tok_score_dir=-1).c())) == 2


def test_gather_joint_validation(lib):
    c = ctypes.byref(dims().c())

    def call(k=2, bt=64, base=10000.0, ci=A, q=A, kq=A, qj=A, kp=None, vp=None, dd=c):
        return lib.pd_gather_joint(dd, k, bt, ci, A, q, A, A, A, kq, A, base, qj, A, A, kp, vp, None)

    assert call(dd=None) == 1
    assert call(k=0) == 2
    assert call(k=5) == 2            # top_k > N
    assert call(bt=0) == 2
    assert call(bt=129) == 2         # tok_budget > C
    assert call(base=-1.0) == 2
    assert call(base=float("nan")) == 2
    assert call(base=float("inf")) == 2
    assert call(ci=None) == 1
    assert call(q=None) == 1
    assert call(kq=None) == 1
    assert call(qj=None) == 1
    assert call(qj=MIS) == 4
    assert call(kp=A) == 1           # one of k_pref / v_pref
    assert call(vp=A) == 1
    assert call(kp=A, vp=MIS) == 4
    assert call(dd=ctypes.byref(dims(head_dim=96).c())) == 3


def test_mfma_probe_validation(lib):
    assert lib.pd_mfma_rate_probe(0, 10, A, None) == 2
    assert lib.pd_mfma_rate_probe(4, 0, A, None) == 2
    assert lib.pd_mfma_rate_probe(4, 10, None, None) == 1
    assert lib.pd_mfma_rate_probe(4, 10, MIS, None) == 4


def test_size_queries():
    d = dims(batch=2, n_chunks=3, chunk_len=100, n_heads_kv=2, n_heads_q=4, head_dim=128, dtype=PD_BF16)
    assert _lib.pd_cache_bytes(d) == 2 * 3 * 2 * 101 * 128 * 2
    d32 = dims(dtype=PD_FP32)
    assert _lib.pd_cache_bytes(d32) == 1 * 4 * 4 * 129 * 64 * 4
    assert _lib.pd_workspace_bytes(dims(batch=0), 0, 0, 0, 0) == 0
    assert _lib.pd_workspace_bytes(d, 0, 0, 0, 0) >= 2 * 3 * 4 * (100 + 16 + 16 + 32) * 4
    # One shard needs no decode workspace; S shards need S partial outputs.
    assert _lib.pd_workspace_bytes(d, 2, 50, 1, 2) == 0
    assert _lib.pd_workspace_bytes(d, 2, 50, 3, 2) >= 3 * 2 * 4 * 32 * 129 * 4
    # The automatic shard count never exceeds the KV tile count.
    for k, bt in [(1, 1), (2, 50), (3, 100)]:
        s = _lib.pd_decode_splits(d, k, bt, 0, 0)
        assert 1 <= s <= max(1, -(-(k * (1 + bt) + 32) // 64))


def test_binding_raises_on_error():
    with pytest.raises(PdError) as ei:
        _lib._check(2)
    assert ei.value.status == 2


def test_error_message_is_thread_local(lib):
    """Each thread reads the message of its own last failure, whatever another
    thread failed with in between."""
    import threading
    bar = threading.Barrier(2)
    out = {}

    def first():
        try:
            out["a_status"] = prefill(dims(), q_pre=None)
            bar.wait()
            bar.wait()
            out["a"] = lib.pd_last_error_message()
        except Exception as e:   # reported below
            out["a_err"] = e

    def second():
        try:
            bar.wait()
            out["b_status"] = prefill(dims(batch=0))
            out["b"] = lib.pd_last_error_message()
            bar.wait()
        except Exception as e:
            out["b_err"] = e

    ts = [threading.Thread(target=first), threading.Thread(target=second)]
    for t in ts:
        t.start()
    for t in ts:
        t.join(30)
    assert "a_err" not in out and "b_err" not in out, out
    assert out["a_status"] == 1 and out["b_status"] == 2
    assert b"q_pre" in out["a"] and b"batch" not in out["a"]
    assert b"batch" in out["b"]
