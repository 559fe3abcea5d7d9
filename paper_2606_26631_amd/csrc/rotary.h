// Device helpers shared by the kernels that rotate keys: 16-byte accesses,
// double -> bfloat16 rounding and the rotation of one pair of chunks.
#pragma once

#include <cmath>
#include <cstdint>

#include <hip/hip_runtime.h>

namespace prcr {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load_nt(const void *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
__device__ __forceinline__ void store_nt(void *p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p));
}

// Round a double to bfloat16, to nearest with ties to even, returned in the low
// 16 bits.  The double is first rounded to float with round-to-odd (truncate
// toward zero and force the last bit on when inexact); float has more than two
// extra bits over bfloat16, so the following float -> bfloat16 round to nearest
// even gives the correctly rounded result of the original double.
__device__ __forceinline__ uint32_t bf16_from_double(double y) {
  const float f = static_cast<float>(y);
  const double back = static_cast<double>(f);
  uint32_t u = __float_as_uint(f);
  u -= (fabs(back) > fabs(y)) ? 1u : 0u;    // rounded away from zero: step back
  u |= (back != y) ? 1u : 0u;               // inexact: force the sticky bit
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return (y != y) ? 0x7FC0u : r;
}

template <typename T>
struct Store;

// float32 storage: a 16-byte chunk holds 4 elements.
template <>
struct Store<float> {
  static constexpr int kPerChunk = 4;
  __device__ static __forceinline__ void rotate(u32x4 lo, u32x4 hi, const double *c,
                                                const double *s, u32x4 &out_lo, u32x4 &out_hi) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double a = static_cast<double>(__uint_as_float(lo[q]));
      const double b = static_cast<double>(__uint_as_float(hi[q]));
      out_lo[q] = __float_as_uint(static_cast<float>(a * c[q] - b * s[q]));
      out_hi[q] = __float_as_uint(static_cast<float>(b * c[q] + a * s[q]));
    }
  }
};

// bfloat16 storage (bit patterns in uint16_t): a 16-byte chunk holds 8 elements.
template <>
struct Store<uint16_t> {
  static constexpr int kPerChunk = 8;
  __device__ static __forceinline__ void rotate(u32x4 lo, u32x4 hi, const double *c,
                                                const double *s, u32x4 &out_lo, u32x4 &out_hi) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const double a0 = static_cast<double>(__uint_as_float(lo[q] << 16));
      const double a1 = static_cast<double>(__uint_as_float(lo[q] & 0xFFFF0000u));
      const double b0 = static_cast<double>(__uint_as_float(hi[q] << 16));
      const double b1 = static_cast<double>(__uint_as_float(hi[q] & 0xFFFF0000u));
      const int e0 = 2 * q, e1 = 2 * q + 1;
      const uint32_t l0 = bf16_from_double(a0 * c[e0] - b0 * s[e0]);
      const uint32_t l1 = bf16_from_double(a1 * c[e1] - b1 * s[e1]);
      const uint32_t h0 = bf16_from_double(b0 * c[e0] + a0 * s[e0]);
      const uint32_t h1 = bf16_from_double(b1 * c[e1] + a1 * s[e1]);
      out_lo[q] = l0 | (l1 << 16);
      out_hi[q] = h0 | (h1 << 16);
    }
  }
};

}  // namespace
}  // namespace prcr
