"""MI355X-native Reformer LSH attention (arXiv:2001.04451).

The compute path is the C-ABI library ``liblsh.so`` built from ``csrc/``
(HIP kernels for gfx950); ``lsh`` is its thin Python binding and
``workloads`` draws the seeded synthetic inputs.  Importing the package
loads nothing; ``paper_2001_04451_amd.lsh`` loads the library on first use.
"""
