"""DQGAN oracle: a plain, slow CPU implementation of one iteration of the
paper's distributed OMD loop with error feedback (Algorithm 2 of
arXiv:2010.13359) and of the compressors it uses (Section 2.4, Theorems 1-2,
Appendix A).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the GPU library (``paper_2010_13359_amd``) and neither imports the
other.
"""
