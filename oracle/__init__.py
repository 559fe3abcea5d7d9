"""CPU oracle for the PRCR rebinding path (test infrastructure only).

Only the tests, the package smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the GPU path.
"""
from .prcr_oracle import *  # noqa: F401,F403
from .prcr_oracle import (MODES, ERR_INDEX, ERR_CAPACITY, ERR_BLOCK, inv_freq, pair_axis,
                          reassign, reassign_batch, rotate_keys, f64_to_bf16_bits,
                          bf16_bits_to_f64, storage_to_f64, f64_to_storage, store_raw,
                          rebind_inject, rebind_entry, rebind_row, slot_of, prefill_capture, decode_attention, cache_rows)
