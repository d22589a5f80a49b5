"""ABCD (Alpha-Composited Block Coordinate Descent) active-block step on MI355X.

The GPU path lives in libabcd.so (hand-written HIP for gfx950, C ABI in
include/abcd.h); `api` is its torch binding and `step` a buffer-reusing driver
of one active-block step. `camera` and `synthetic` hold plain inputs.
"""
__version__ = "0.1.0"
