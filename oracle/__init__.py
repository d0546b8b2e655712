"""CPU oracle for the ARCHead packed LM-head forward (TEST INFRASTRUCTURE).

This package is a plain, slow, fp64 NumPy implementation of what the packed
head computes, written from the paper (ARCHead, arXiv 2608.02703) and from the
packed layout described in ``include/archead.h``.  It exists to check the HIP
path, and only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import it.  The product path never calls it, and it
shares no code with the HIP library: it unpacks the layout itself, forms the
dequantised dense head in fp64 and takes the matrix products with BLAS.

Modules
  layout     INT4 nibble layout, fp16 / bf16 bit decoding
  head       dense head W_hat = W_res + U_c V_c + A B, logits, CE, argmax
  bytes      persistent-byte accounting (sum of numel x element size)
  construct  damped covariance, metric transform, correction fit by exact SVD
  metrics    PPL and relative PPL; logit fidelity (KL, top-k agreement, MSE)
"""
from . import layout, head, bytes as bytes_, construct, metrics  # noqa: F401
