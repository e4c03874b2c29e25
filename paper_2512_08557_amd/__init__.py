"""MI355X (gfx950) delta-scatter convolution with temporal data recycling.

The hot path (changed-cell detection, delta packing, MFMA contraction with
persistent per-layer maps, activation-delta epilogue and change-list
propagation) lives in libsscater.so, built from csrc/ by build.py; this
package is its ctypes binding.
"""
from .engine import (BF16, E_DEVICE, E_HIP, E_INVALID_ARG, E_OUT_OF_MEMORY, E_OVERFLOW, EXPORTS, F32, OK,
                     Engine, SscaterError, lib, LIB_PATH)

__all__ = ["Engine", "SscaterError", "lib", "LIB_PATH", "EXPORTS", "OK", "E_INVALID_ARG", "E_OUT_OF_MEMORY",
           "E_HIP", "E_OVERFLOW", "E_DEVICE", "F32", "BF16"]
