"""PRCR position-rebinding cache reuse on AMD MI355X (gfx950).

The work runs in hand-written HIP kernels behind the C ABI of include/prcr.h
(libprcr.so, built in this directory); this package is the thin Python binding.
"""
from .binding import (DERR_BLOCK, DERR_CAPACITY, DERR_INDEX, DERR_OFFSETS, DERR_RANGE, MODES,
                      Cache, Memory, PrcrError, Rope, decode_attention, decode_attention_static,
                      decode_workspace_bytes, lib,
                      prefill_capture, reassign_coords, rebind_inject, revisit, store_raw)

__all__ = ["Cache", "Memory", "Rope", "PrcrError", "lib", "store_raw", "prefill_capture",
           "decode_attention", "decode_attention_static", "decode_workspace_bytes", "reassign_coords",
           "rebind_inject", "revisit", "MODES", "DERR_INDEX", "DERR_CAPACITY", "DERR_BLOCK", "DERR_OFFSETS",
           "DERR_RANGE"]
