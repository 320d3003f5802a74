"""PRQuant (Permutation Residual Quantization) MXFP4 hot path for MI355X (gfx950).

The compute lives in ``libprq.so`` (hand-written HIP kernels and a C ABI, see
``include/prq.h``).  ``paper_2609_22106_amd.prq`` is the ctypes binding with
the same call names; importing it loads the library and fails loudly when the
library has not been built.  ``paper_2609_22106_amd.inputs`` holds the seeded
synthetic workloads and does not load the library.
"""

__all__ = ["prq", "inputs", "build"]


def __getattr__(name):  # lazy: importing ``inputs`` must not load the library
    if name in ("prq", "inputs", "build"):
        import importlib
        return importlib.import_module(f"{__name__}.{name}")
    raise AttributeError(name)
