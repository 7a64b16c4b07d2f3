"""MI355X (gfx950) implementation of the per-iteration gradient-compression
path of DQGAN (arXiv:2010.13359, Algorithm 2): error-feedback accumulate,
delta-approximate compressors (scaled sign, s-level stochastic quantizer,
top-k), message packing, server average and the optimistic-mirror-descent
update with the per-worker extrapolated point.

The computation lives in the HIP library ``libdqgan.so`` behind the C ABI of
``include/dqgan.h``; ``dqgan`` is its Python binding.
"""
from . import dqgan  # noqa: F401
