"""MI355X (gfx950) block-sparse attention path of Prefilling-dLLM.

The compute lives in ``libpd.so`` (HIP kernels behind the C ABI of
include/pd.h); ``_lib`` is its ctypes binding, ``synth`` draws the seeded
synthetic workloads, ``build`` compiles the library.
"""

__all__ = ["_lib", "synth", "build"]
