"""Test helper: the fp64 oracle on a pool of worker processes, for the full-size parity samples.

The parent writes the arrays the workers need (the inputs of the checked
sequences and the GPU's outputs for them, as float32 host copies: bf16 and fp32
values are exact in float32) to one file in a temporary directory; every worker
maps it read-only (page cache, no size limit of a shared-memory mount) and
evaluates oracle units on it.  A prefill unit returns only its
error margin against the GPU output and its Eq. 5 head term, so nothing large
crosses the process boundary.  Workers use one BLAS thread each and never touch
the GPU.
"""

import concurrent.futures as cf
import multiprocessing as mp
import os
import shutil
import tempfile

import numpy as np

WORKERS = max(1, min(len(os.sched_getaffinity(0)), 16))   # one GPU's share of the host

_S = {}   # worker state: name -> array view of the shared block


def _attach(path, layout):
    for key, (off, shape) in layout.items():
        _S[key] = np.memmap(path, dtype=np.float32, mode="r", offset=off, shape=shape)


def _init(name, layout):
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)
    _attach(name, layout)


def _prefill_unit(b, n, h, q_len, tol, out_rounding):
    """Oracle prefill unit (b, n, h) against the GPU output; returns (b, n, h, margin, e_head) where margin
    = max(err - bound) over the unit (<= 0 passes) with bound = tol + out_rounding * |O_ref|."""
    import oracle
    u = oracle.prefill_unit_ref(_S["q_pre"], _S["k_pre"], _S["v_pre"], _S["q_qm"], _S["k_qm"], _S["v_qm"], b, n, h,
                                q_len)
    got = _S["o"][b, n, :, h, :].astype(np.float64)
    margin = float(np.max(np.abs(got - u["o"]) - (tol + out_rounding * np.abs(u["o"]))))
    return b, n, h, margin, u["e_head"]


class OraclePool:
    """A file of float32 copies of `arrays` (dict name -> numpy array) and a process pool mapping it."""

    def __init__(self, arrays):
        layout, off = {}, 0
        for k, a in arrays.items():
            layout[k] = (off, a.shape)
            off += (a.size * 4 + 255) // 256 * 256
        self.dir = tempfile.mkdtemp(prefix="oracle_pool_", dir="/tmp")
        path = os.path.join(self.dir, "arrays.f32")
        mm = np.memmap(path, dtype=np.float32, mode="w+", shape=(max(off, 256) // 4,))
        for k, a in arrays.items():
            o, shape = layout[k]
            mm[o // 4: o // 4 + a.size] = np.asarray(a, dtype=np.float32).reshape(-1)
        mm.flush()
        del mm
        saved = {v: os.environ.get(v) for v in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
        for v in saved:
            os.environ[v] = "1"   # inherited by the spawned workers before they import numpy
        try:
            self.ex = cf.ProcessPoolExecutor(WORKERS, mp_context=mp.get_context("spawn"), initializer=_init,
                                             initargs=(path, layout))
            list(self.ex.map(abs, range(WORKERS)))   # start every worker while the variables are set
        finally:
            for v, old in saved.items():
                if old is None:
                    os.environ.pop(v, None)
                else:
                    os.environ[v] = old

    def prefill_units(self, units, q_len, tol, out_rounding):
        futs = [self.ex.submit(_prefill_unit, b, n, h, q_len, tol, out_rounding) for b, n, h in units]
        return [f.result() for f in futs]

    def close(self):
        self.ex.shutdown(wait=True)
        shutil.rmtree(self.dir, ignore_errors=True)

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
