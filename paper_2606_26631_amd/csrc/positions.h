// Position reassignment arithmetic (Sec. 3.2, Eq. (8)-(10)), shared by the
// stand-alone reassignment kernel and the fused revisit kernel.
#pragma once

#include <climits>
#include <cmath>
#include <cstdint>

#include "prcr.h"

namespace prcr {

constexpr double kExactLimit = 4503599627370496.0;   // 2^52

// PCR along one axis: A + (L + 1)(1 + (K - 1) u)/(K + 1) with A = p_txt - L
// (leftward, Eq. (10)) or A = p_txt + 1 (rightward), u = (c - lo)/(hi - lo), or
// u = 1/2 when hi == lo.  Formed as an integer numerator and denominator and
// divided once in double, which is the correctly rounded value of the rational
// while both stay below 2^52; beyond that a close double approximation is
// returned and *range_bad is set.
__device__ __forceinline__ double pcr_position(int64_t A, int64_t L, int64_t K, int64_t lo,
                                               int64_t hi, int64_t c, bool *range_bad) {
  const int64_t span = hi - lo;
  if (span <= 0) {
    // u = 1/2:  A + (L + 1)/2 = (2A + L + 1) / 2
    const double mag = 2.0 * fabs(static_cast<double>(A)) + static_cast<double>(L + 1);
    if (mag >= kExactLimit) {
      *range_bad = true;
      return static_cast<double>(A) + 0.5 * static_cast<double>(L + 1);
    }
    return static_cast<double>(2 * A + L + 1) / 2.0;
  }
  const double kd = static_cast<double>(K + 1) * static_cast<double>(span);
  const double mag = (fabs(static_cast<double>(A)) + static_cast<double>(L + 1)) * kd;
  if (mag >= kExactLimit || kd >= kExactLimit) {
    *range_bad = true;
    const double frac = static_cast<double>(L + 1) *
                        (static_cast<double>(span) +
                         static_cast<double>(K - 1) * static_cast<double>(c - lo)) / kd;
    return static_cast<double>(A) + frac;
  }
  const int64_t den = (K + 1) * span;
  const int64_t num = A * den + (L + 1) * (span + (K - 1) * (c - lo));
  return static_cast<double>(num) / static_cast<double>(den);
}

// New coordinate of the token of rank j (0-based, selection order) among K
// selected tokens along an axis whose valid coordinates span [lo, hi].
__device__ __forceinline__ double reassigned(int mode, int64_t p_txt, int64_t L, int64_t K,
                                             int64_t j, int64_t lo, int64_t hi, int64_t c,
                                             bool *range_bad) {
  switch (mode) {
    case PRCR_MODE_SHIFT:
      return static_cast<double>(p_txt + 1 + (c - lo));
    case PRCR_MODE_IDENTITY:
      return static_cast<double>(c);
    case PRCR_MODE_LPA:
      return static_cast<double>(p_txt + j + 1);
    case PRCR_MODE_UIR: {
      const double mag = fabs(static_cast<double>(p_txt)) * static_cast<double>(K + 1) + K + 1;
      if (mag >= kExactLimit) {
        *range_bad = true;
        return static_cast<double>(p_txt) + static_cast<double>(j + 1) / static_cast<double>(K + 1);
      }
      return static_cast<double>(p_txt * (K + 1) + j + 1) / static_cast<double>(K + 1);
    }
    case PRCR_MODE_PCR_RIGHT:
      return pcr_position(p_txt + 1, L, K, lo, hi, c, range_bad);
    default:
      return pcr_position(p_txt - L, L, K, lo, hi, c, range_bad);
  }
}

// Next text position after the revisit.  any_valid: at least one selected token
// had a valid index; max_span: the largest hi - lo over the three axes.
__device__ __forceinline__ int64_t next_text_position(int mode, int64_t p_txt, int64_t K,
                                                      bool any_valid, int64_t max_span) {
  if (mode == PRCR_MODE_LPA) return p_txt + K + 1;
  if (mode == PRCR_MODE_SHIFT && any_valid) return p_txt + 2 + max_span;
  return p_txt + 1;
}

// The next text position as the int32 the ABI returns: a value outside the
// int32 range is saturated to its nearest end and *range_bad is set (the caller
// then reports PRCR_DERR_RANGE), never wrapped.
__device__ __forceinline__ int32_t next_pos_int32(int64_t next, bool *range_bad) {
  if (next > INT32_MAX) {
    *range_bad = true;
    return INT32_MAX;
  }
  if (next < INT32_MIN) {
    *range_bad = true;
    return INT32_MIN;
  }
  return static_cast<int32_t>(next);
}

}  // namespace prcr
