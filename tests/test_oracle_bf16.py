"""Pins for the oracle's float64 -> bfloat16 round-to-nearest-even.

References: torch's float32 -> bfloat16 cast (a library RNE) on inputs that are
exactly float32, exhaustive enumeration of bf16 values, and the tie rule checked
at exact midpoints and one float64 step away from them.
"""
import numpy as np
import torch

from oracle import bf16_bits_to_f64, f64_to_bf16_bits


def _all_finite_bf16():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = bf16_bits_to_f64(bits)
    keep = np.isfinite(vals)
    return bits[keep], vals[keep]


def test_exact_values_round_to_themselves():
    bits, vals = _all_finite_bf16()
    out = f64_to_bf16_bits(vals)
    # -0.0 and +0.0 both keep their sign bit
    assert np.array_equal(out, bits)


def test_matches_torch_cast_on_float32_inputs():
    rng = np.random.default_rng(3)
    with np.errstate(over="ignore"):            # draws beyond the float32 range become inf
        x = np.concatenate([
            rng.standard_normal(200_000).astype(np.float32),
            (rng.standard_normal(50_000) * 1e-38).astype(np.float32),   # bf16 subnormal range
            (rng.standard_normal(50_000) * 3e38).astype(np.float32),    # near overflow
            rng.integers(0, 1 << 32, 200_000, dtype=np.uint64).astype(np.uint32).view(np.float32),
        ])
    x = x[np.isfinite(x)]
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    out = f64_to_bf16_bits(x.astype(np.float64))
    assert np.array_equal(out, ref)


def test_ties_to_even_and_off_tie_inputs():
    bits, vals = _all_finite_bf16()
    pos = (vals > 0) & np.isfinite(vals)
    b, v = bits[pos].astype(np.int64), vals[pos]
    order = np.argsort(v)
    b, v = b[order], v[order]
    lo, hi = v[:-1], v[1:]
    blo, bhi = b[:-1], b[1:]
    mid = (lo + hi) / 2                      # exact in float64
    even = np.where(blo % 2 == 0, blo, bhi)
    assert np.array_equal(f64_to_bf16_bits(mid).astype(np.int64), even)
    up = np.nextafter(mid, np.inf)
    dn = np.nextafter(mid, -np.inf)
    assert np.array_equal(f64_to_bf16_bits(up).astype(np.int64), bhi)
    assert np.array_equal(f64_to_bf16_bits(dn).astype(np.int64), blo)
    # and symmetrically for negative values
    assert np.array_equal(f64_to_bf16_bits(-up).astype(np.int64), bhi | 0x8000)


def test_special_values():
    out = f64_to_bf16_bits(np.array([np.inf, -np.inf, np.nan, 1e300, -1e300, 0.0, -0.0, 1e-300]))
    assert out.tolist() == [0x7F80, 0xFF80, 0x7FC0, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x0000]
