"""MI355X-native E2-TTT chunk-parallel fast-weight update (arxiv 2608.21308).

The compute path is a HIP shared library (``libe2ttt.so``, C ABI declared in
``include/e2ttt.h``); ``paper_2608_21308_amd.e2ttt`` is a thin ctypes binding
over it.  ``workloads`` holds the seeded synthetic input recipes.
"""
