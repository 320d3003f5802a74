"""CPU oracle for PRQuant (Permutation Residual Quantization), arXiv 2609.22106.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
anything in this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It is a plain, slow, obviously
correct NumPy implementation, in float64 wherever the paper does not fix the
precision, written from the paper's definitions:

* ``oracle.mxfp4``   -- the MXFP4 quantize/dequantize operator Q(.) that the
  paper uses throughout (Sec. 1, and Eq. 2 where Q is introduced; the format is
  the OCP Microscaling one the paper cites).
* ``oracle.prquant`` -- offline calibration and export (Algorithm 1 for one
  alpha: scaling, top-k column selection, permutation, tail residual of Eq. 2,
  augmented weight of Eq. 3), the activation side of Eq. 3 (online copy,
  Sec. "Activation tail construction"), the augmented GEMM of Eq. 3, its
  grouped (MoE expert) form, the unquantized identity of Eq. 1 and the
  normalized reconstruction error used for alpha selection and the ablation.

It shares no code, header, table or helper with the HIP path.  Inputs come from
the seeded generators in ``paper_2609_22106_amd.inputs`` (random draws only, no
arithmetic of the method).
"""
from . import mxfp4, prquant  # noqa: F401
