"""ctypes binding of ``libpd.so`` (the C ABI declared in include/pd.h).

Argument marshalling only: torch tensors are passed as device pointers, the
stream as its ``hipStream_t`` handle; every step of the path runs in the HIP
kernels.  If the library is missing this module raises -- there is no CPU
fallback.
"""

import ctypes
import os
from dataclasses import dataclass

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libpd.so")

PD_BF16, PD_FP32 = 0, 1
STATUS = {0: "PD_OK", 1: "PD_ERR_NULL_PTR", 2: "PD_ERR_BAD_DIMS", 3: "PD_ERR_UNSUPPORTED",
          4: "PD_ERR_MISALIGNED", 5: "PD_ERR_WORKSPACE", 6: "PD_ERR_HIP"}

EXPORTS = ["pd_prefill_chunks", "pd_score_select", "pd_sparse_decode_attn", "pd_cache_bytes",
           "pd_workspace_bytes", "pd_decode_splits", "pd_status_string", "pd_last_error_message",
           "pd_version", "pd_mfma_rate_probe", "pd_score_select_static", "pd_gather_selected",
           "pd_sparse_decode_attn_compact", "pd_compact_workspace_bytes", "pd_select_ranked",
           "pd_gather_joint", "pd_score_select_noalloc"]


class PdError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class PdDims(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("n_chunks", ctypes.c_int32), ("chunk_len", ctypes.c_int32),
        ("q_len", ctypes.c_int32), ("m_len", ctypes.c_int32), ("dec_len", ctypes.c_int32),
        ("n_heads_q", ctypes.c_int32), ("n_heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32), ("sm_scale", ctypes.c_float), ("qm_per_chunk", ctypes.c_int32),
        ("out_fp32", ctypes.c_int32), ("tok_score_dir", ctypes.c_int32),
    ]


@dataclass
class Dims:
    """Problem sizes in the paper's notation (Section 5): B, N, C, L_q, L_m, L_d, heads, d."""
    batch: int
    n_chunks: int
    chunk_len: int
    q_len: int
    m_len: int
    dec_len: int
    n_heads_q: int
    n_heads_kv: int
    head_dim: int
    dtype: int = PD_BF16
    sm_scale: float = 0.0
    qm_per_chunk: int = 0
    out_fp32: int = 0
    tok_score_dir: int = 0

    @property
    def seq_len(self):
        """S_c = 1 + C + L_q + L_m, rows of one chunk sequence."""
        return 1 + self.chunk_len + self.q_len + self.m_len

    def c(self):
        return PdDims(self.batch, self.n_chunks, self.chunk_len, self.q_len, self.m_len, self.dec_len,
                      self.n_heads_q, self.n_heads_kv, self.head_dim, self.dtype, self.sm_scale,
                      self.qm_per_chunk, self.out_fp32, self.tok_score_dir)


_lib = None


def load(path: str = LIB_PATH):
    """Load libpd.so once and declare the signatures; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library not built: {path} (run __graft_entry__.build())")
    # torch ships its own HIP runtime with the same soname; loading torch first
    # makes libpd.so bind to that one copy, so streams and device pointers the
    # caller gets from torch belong to the runtime that launches the kernels.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, sz, i32, fp = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_void_p
    dp = ctypes.POINTER(PdDims)
    lib.pd_prefill_chunks.argtypes = [dp] + [vp] * 13 + [vp, sz, vp]
    lib.pd_prefill_chunks.restype = ctypes.c_int
    lib.pd_score_select.argtypes = [dp, i32, i32, vp, fp, fp, vp, vp, fp, vp, sz, vp]
    lib.pd_score_select.restype = ctypes.c_int
    lib.pd_sparse_decode_attn.argtypes = [dp, i32, i32] + [vp] * 9 + [i32, vp, fp, i32, vp, sz, vp]
    lib.pd_sparse_decode_attn.restype = ctypes.c_int
    lib.pd_cache_bytes.argtypes = [dp]
    lib.pd_cache_bytes.restype = sz
    lib.pd_workspace_bytes.argtypes = [dp, i32, i32, i32, i32]
    lib.pd_workspace_bytes.restype = sz
    lib.pd_decode_splits.argtypes = [dp, i32, i32, i32, i32]
    lib.pd_decode_splits.restype = i32
    lib.pd_status_string.argtypes = [ctypes.c_int]
    lib.pd_status_string.restype = ctypes.c_char_p
    lib.pd_last_error_message.argtypes = []
    lib.pd_last_error_message.restype = ctypes.c_char_p
    lib.pd_select_ranked.argtypes = [dp, i32, i32, fp, i32, fp, vp, vp, vp]
    lib.pd_select_ranked.restype = ctypes.c_int
    lib.pd_score_select_noalloc.argtypes = [dp, i32, i32, vp, fp, fp, vp, vp, fp, vp]
    lib.pd_score_select_noalloc.restype = ctypes.c_int
    lib.pd_score_select_static.argtypes = [dp, i32, i32, vp, fp, fp, vp, vp, fp, vp, sz, vp]
    lib.pd_score_select_static.restype = ctypes.c_int
    lib.pd_gather_selected.argtypes = [dp, i32, i32] + [vp] * 6 + [vp]
    lib.pd_gather_selected.restype = ctypes.c_int
    lib.pd_gather_joint.argtypes = [dp, i32, i32] + [vp] * 8 + [ctypes.c_double] + [vp] * 6
    lib.pd_gather_joint.restype = ctypes.c_int
    lib.pd_sparse_decode_attn_compact.argtypes = [dp, i32] + [vp] * 7 + [i32, vp, fp, i32, vp, sz, vp]
    lib.pd_sparse_decode_attn_compact.restype = ctypes.c_int
    lib.pd_compact_workspace_bytes.argtypes = [dp, i32, i32]
    lib.pd_compact_workspace_bytes.restype = sz
    lib.pd_mfma_rate_probe.argtypes = [i32, i32, vp, vp]
    lib.pd_mfma_rate_probe.restype = ctypes.c_int
    lib.pd_version.argtypes = []
    lib.pd_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _ptr(t):
    """Device pointer of a tensor (or None / an int address)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensors passed to the HIP library must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return stream if isinstance(stream, int) else stream.cuda_stream


def _check(status):
    if status != 0:
        raise PdError(status, load().pd_last_error_message().decode())


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def pd_cache_bytes(dims: Dims) -> int:
    return load().pd_cache_bytes(ctypes.byref(dims.c()))


def pd_workspace_bytes(dims: Dims, top_k=0, tok_budget=0, num_splits=0, which=0) -> int:
    return load().pd_workspace_bytes(ctypes.byref(dims.c()), top_k, tok_budget, num_splits, which)


def pd_decode_splits(dims: Dims, top_k, tok_budget, n_static, num_splits=0) -> int:
    return load().pd_decode_splits(ctypes.byref(dims.c()), top_k, tok_budget, n_static, num_splits)


def pd_prefill_chunks(dims: Dims, q_pre, k_pre, v_pre, q_qm, k_qm, v_qm, o, k_cache, v_cache,
                      tok_score, tok_rank, key_mean, workspace, stream=None, chunk_score=None):
    """Stage (a) for one layer (see include/pd.h); chunk_score (B, N) fp32 or None."""
    _check(load().pd_prefill_chunks(
        ctypes.byref(dims.c()), _ptr(q_pre), _ptr(k_pre), _ptr(v_pre), _ptr(q_qm), _ptr(k_qm), _ptr(v_qm),
        _ptr(o), _ptr(k_cache), _ptr(v_cache), _ptr(tok_score), _ptr(tok_rank), _ptr(key_mean),
        _ptr(chunk_score), _ptr(workspace), _nbytes(workspace), _stream(stream)))


def pd_select_ranked(dims: Dims, top_k, tok_budget, chunk_score, lowest, tok_rank, chunk_idx, tok_slot,
                     stream=None):
    """Top-K chunks by given scores (the lowest when lowest=1) and their kept tokens (see include/pd.h)."""
    _check(load().pd_select_ranked(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(chunk_score), int(lowest), _ptr(tok_rank),
        _ptr(chunk_idx), _ptr(tok_slot), _stream(stream)))


def pd_score_select(dims: Dims, top_k, tok_budget, q_dec, key_mean, tok_rank, chunk_idx, tok_slot,
                    chunk_score, workspace, stream=None):
    """Stage (b) for one layer and step (see include/pd.h)."""
    _check(load().pd_score_select(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(q_dec), _ptr(key_mean), _ptr(tok_rank),
        _ptr(chunk_idx), _ptr(tok_slot), _ptr(chunk_score), _ptr(workspace), _nbytes(workspace),
        _stream(stream)))


def pd_score_select_noalloc(dims: Dims, top_k, tok_budget, q_dec, key_mean, tok_rank, chunk_idx, tok_slot,
                            chunk_score=None, stream=None):
    """Stage (b) without a workspace: scratch in the library's static per-GPU array (see include/pd.h)."""
    _check(load().pd_score_select_noalloc(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(q_dec), _ptr(key_mean), _ptr(tok_rank),
        _ptr(chunk_idx), _ptr(tok_slot), _ptr(chunk_score), _stream(stream)))


def pd_sparse_decode_attn(dims: Dims, top_k, tok_budget, q_dec, k_dec, v_dec, k_cache, v_cache,
                          chunk_idx, tok_slot, k_static, v_static, n_static, o_dec, lse_dec,
                          num_splits, workspace, stream=None):
    """Stage (c) for one layer and step (see include/pd.h)."""
    _check(load().pd_sparse_decode_attn(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(q_dec), _ptr(k_dec), _ptr(v_dec),
        _ptr(k_cache), _ptr(v_cache), _ptr(chunk_idx), _ptr(tok_slot), _ptr(k_static), _ptr(v_static),
        n_static, _ptr(o_dec), _ptr(lse_dec), num_splits, _ptr(workspace), _nbytes(workspace),
        _stream(stream)))


def pd_score_select_static(dims: Dims, top_k, tok_budget, q_qm, key_mean, tok_rank, chunk_idx, tok_slot,
                           chunk_score, workspace, stream=None):
    """Static-selection mode: selection from the pseudo-label rows of q_qm (see include/pd.h)."""
    _check(load().pd_score_select_static(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(q_qm), _ptr(key_mean), _ptr(tok_rank),
        _ptr(chunk_idx), _ptr(tok_slot), _ptr(chunk_score), _ptr(workspace), _nbytes(workspace),
        _stream(stream)))


def pd_gather_selected(dims: Dims, top_k, tok_budget, k_cache, v_cache, chunk_idx, tok_slot, k_sel, v_sel,
                       stream=None):
    """Static-selection mode: copy the kept rows into contiguous buffers (see include/pd.h)."""
    _check(load().pd_gather_selected(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(k_cache), _ptr(v_cache), _ptr(chunk_idx),
        _ptr(tok_slot), _ptr(k_sel), _ptr(v_sel), _stream(stream)))


def pd_gather_joint(dims: Dims, top_k, tok_budget, chunk_idx, tok_slot, q_pre, k_cache, v_cache, q_qm, k_qm,
                    v_qm, rope_base, q_joint, k_joint, v_joint, k_pref=None, v_pref=None, stream=None):
    """Full-mask mode: joint rows [kept rows ; query rows] at continuous positions (see include/pd.h)."""
    _check(load().pd_gather_joint(
        ctypes.byref(dims.c()), top_k, tok_budget, _ptr(chunk_idx), _ptr(tok_slot), _ptr(q_pre), _ptr(k_cache),
        _ptr(v_cache), _ptr(q_qm), _ptr(k_qm), _ptr(v_qm), float(rope_base), _ptr(q_joint), _ptr(k_joint),
        _ptr(v_joint), _ptr(k_pref), _ptr(v_pref), _stream(stream)))


def pd_sparse_decode_attn_compact(dims: Dims, n_sel, q_dec, k_dec, v_dec, k_sel, v_sel, k_static, v_static,
                                  n_static, o_dec, lse_dec, num_splits, workspace, stream=None):
    """Stage (c) over a compact prefix buffer (see include/pd.h)."""
    _check(load().pd_sparse_decode_attn_compact(
        ctypes.byref(dims.c()), n_sel, _ptr(q_dec), _ptr(k_dec), _ptr(v_dec), _ptr(k_sel), _ptr(v_sel),
        _ptr(k_static), _ptr(v_static), n_static, _ptr(o_dec), _ptr(lse_dec), num_splits, _ptr(workspace),
        _nbytes(workspace), _stream(stream)))


def pd_compact_workspace_bytes(dims: Dims, n_sel, num_splits=0) -> int:
    return load().pd_compact_workspace_bytes(ctypes.byref(dims.c()), n_sel, num_splits)


def pd_mfma_rate_probe(n_workgroups, iters, sink, stream=None):
    """Launch the MFMA-rate diagnostic (n_workgroups * 4 * iters * 8 * 32768 FLOP)."""
    _check(load().pd_mfma_rate_probe(n_workgroups, iters, _ptr(sink), _stream(stream)))
