"""Quantized selective-state update for MI355X (gfx950).

A C ABI library (libssmq.so, see include/ssmq.h) with hand-written HIP kernels
for the per-token Mamba state update over a low-precision state cache, rounded
by round-to-nearest, stochastic rounding or the golden-ratio Weyl dither
("Low-Discrepancy Dither for Quantized Recurrent State Caches"). This package
is the thin Python binding (argument marshalling) plus seeded workloads.
"""
from ._binding import (  # noqa: F401
    CODE_BYTES, FORMATS, RULES, SsmqError, conv1d_update, dither_fill, library, replay,
    requantize, state_update,
)

__all__ = ["state_update", "conv1d_update", "requantize", "dither_fill", "replay", "library",
           "SsmqError",
           "RULES",
           "FORMATS", "CODE_BYTES"]
