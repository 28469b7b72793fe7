"""BITCOS ternary GEMV for MI355X (gfx950).

The product is libbitcos.so (C ABI in include/bitcos.h): host packers for the
BITCOS layout (presence bitmap + compacted signs, 2 - z bits per weight) and
two fixed-rate baselines, and hand-written HIP GEMV kernels for all three.
``paper_2609_16338_amd.api`` is the thin Python binding with the same names.
Importing this package does not load the library; ``api`` does, on first
use, and raises if it has not been built.
"""
