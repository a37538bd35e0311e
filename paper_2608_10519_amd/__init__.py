"""SparSTAR hot path for AMD Instinct MI355X (gfx950).

`paper_2608_10519_amd.sparstar` binds the HIP library (libsparstar.so, built by
`python -m paper_2608_10519_amd.build`); the C ABI is include/sparstar.h.
"""
