// Position reassignment for the selected tokens (Sec. 3.2, Eq. (8)-(10)).
//
// One workgroup per sequence: a block-wide min/max over the valid selected
// coordinates (Eq. (8)), then one thread per token writes its new (t, h, w)
// position.  PCR positions are the exact rational of Eq. (9)-(10) over integer
// numerator and denominator, divided once in double precision, which makes the
// value the correctly rounded one and identical on every device.
#include <climits>
#include <cmath>

#include "prcr_internal.h"

namespace prcr {
namespace {

constexpr int kThreads = 256;
constexpr double kExact = 9007199254740992.0;   // 2^53

__device__ __forceinline__ int wave_min(int v) {
  for (int o = kWave / 2; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
  for (int o = kWave / 2; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  return v;
}

// (p_txt - L) + (L + 1)(D + (K - 1)(c - lo)) / ((K + 1) D), or the interval
// centre for a degenerate axis.  Sets *range_bad when the integer rational is
// not exactly representable (then the value is a close double approximation).
__device__ __forceinline__ double pcr_position(int64_t p_txt, int64_t L, int64_t K, int64_t lo,
                                               int64_t hi, int64_t c, bool *range_bad) {
  const int64_t A = p_txt - L;
  int64_t span = hi - lo;
  if (span <= 0) {
    // u = 1/2:  A + (L + 1)/2 = (2A + L + 1) / 2
    const double mag = 2.0 * fabs(static_cast<double>(A)) + static_cast<double>(L + 1);
    if (mag >= kExact) {
      *range_bad = true;
      return static_cast<double>(A) + 0.5 * static_cast<double>(L + 1);
    }
    return static_cast<double>(2 * A + L + 1) / 2.0;
  }
  const double kd = static_cast<double>(K + 1) * static_cast<double>(span);
  const double mag = (fabs(static_cast<double>(A)) + static_cast<double>(L + 1)) * kd;
  if (mag >= kExact * 0.5 || kd >= kExact) {
    *range_bad = true;
    const double frac = static_cast<double>(L + 1) *
                        (static_cast<double>(span) + static_cast<double>(K - 1) * static_cast<double>(c - lo)) /
                        kd;
    return static_cast<double>(A) + frac;
  }
  const int64_t den = (K + 1) * span;
  const int64_t num = A * den + (L + 1) * (span + (K - 1) * (c - lo));
  return static_cast<double>(num) / static_cast<double>(den);
}

__global__ __launch_bounds__(kThreads) void reassign_kernel(const ReassignParams p) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  __shared__ int s_lo[kThreads / kWave][3];
  __shared__ int s_hi[kThreads / kWave][3];
  __shared__ int s_bad[kThreads / kWave];

  const int64_t p_txt = p.p_txt[b];
  const int s0 = p.sel_off[b];
  const int s1 = p.sel_off[b + 1];
  bool offsets_ok = s0 >= 0 && s0 <= s1 && s1 <= p.total_k;
  if (b == 0 && p.sel_off[0] != 0) offsets_ok = false;
  if (b == p.batch - 1 && s1 != p.total_k) offsets_ok = false;
  if (!offsets_ok) {
    if (tid == 0) {
      p.next_pos[b] = static_cast<int32_t>(p_txt + 1);
      if (p.err != nullptr) atomicOr(p.err, PRCR_DERR_OFFSETS);
    }
    // Out-of-range offsets leave this sequence's positions unwritten.
    if (!(s0 >= 0 && s0 <= s1 && s1 <= p.total_k)) return;
  }
  const int K = s1 - s0;
  const int64_t L = p.l_ext;
  const int nvis = min(p.n_visual[b], p.max_visual);
  const int32_t *coords_b = p.coords + static_cast<int64_t>(b) * p.max_visual * 3;

  // Eq. (8): per-axis range over the valid selected tokens.
  int lo[3] = {INT_MAX, INT_MAX, INT_MAX};
  int hi[3] = {INT_MIN, INT_MIN, INT_MIN};
  int bad = 0;
  for (int j = tid; j < K; j += kThreads) {
    const int m = p.sel_idx[s0 + j];
    if (m < 0 || m >= nvis) {
      bad = 1;
      continue;
    }
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const int c = coords_b[3 * m + a];
      lo[a] = min(lo[a], c);
      hi[a] = max(hi[a], c);
    }
  }
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    lo[a] = wave_min(lo[a]);
    hi[a] = wave_max(hi[a]);
  }
  bad = wave_max(bad);
  if (lane == 0) {
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      s_lo[wave][a] = lo[a];
      s_hi[wave][a] = hi[a];
    }
    s_bad[wave] = bad;
  }
  __syncthreads();
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    lo[a] = s_lo[0][a];
    hi[a] = s_hi[0][a];
    for (int w = 1; w < kThreads / kWave; ++w) {
      lo[a] = min(lo[a], s_lo[w][a]);
      hi[a] = max(hi[a], s_hi[w][a]);
    }
  }
  bad = 0;
  for (int w = 0; w < kThreads / kWave; ++w) bad |= s_bad[w];
  const bool any_valid = lo[0] <= hi[0];

  int range_bad = 0;
  for (int j = tid; j < K; j += kThreads) {
    const int m = p.sel_idx[s0 + j];
    double *out = p.new_pos + 3 * static_cast<int64_t>(s0 + j);
    if (m < 0 || m >= nvis) {
      out[0] = out[1] = out[2] = __builtin_nan("");
      continue;
    }
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const int64_t c = coords_b[3 * m + a];
      double v;
      switch (p.mode) {
        case PRCR_MODE_SHIFT:
          v = static_cast<double>(p_txt + 1 + (c - lo[a]));
          break;
        case PRCR_MODE_IDENTITY:
          v = static_cast<double>(c);
          break;
        case PRCR_MODE_LPA:
          v = static_cast<double>(p_txt + j + 1);
          break;
        case PRCR_MODE_UIR: {
          const double mag = fabs(static_cast<double>(p_txt)) * static_cast<double>(K + 1) + K + 1;
          if (mag >= kExact) {
            range_bad = 1;
            v = static_cast<double>(p_txt) + static_cast<double>(j + 1) / static_cast<double>(K + 1);
          } else {
            v = static_cast<double>(p_txt * (K + 1) + j + 1) / static_cast<double>(K + 1);
          }
          break;
        }
        default: {
          bool rb = false;
          v = pcr_position(p_txt, L, K, lo[a], hi[a], c, &rb);
          range_bad |= rb ? 1 : 0;
          break;
        }
      }
      out[a] = v;
    }
  }

  if (tid == 0) {
    int64_t next = p_txt + 1;
    if (p.mode == PRCR_MODE_LPA) {
      next = p_txt + K + 1;
    } else if (p.mode == PRCR_MODE_SHIFT && any_valid) {
      int64_t span = 0;
      for (int a = 0; a < 3; ++a)
        span = max(span, static_cast<int64_t>(hi[a]) - static_cast<int64_t>(lo[a]));
      next = p_txt + 2 + span;
    }
    p.next_pos[b] = static_cast<int32_t>(next);
    if (bad && p.err != nullptr) atomicOr(p.err, PRCR_DERR_INDEX);
  }
  if (range_bad && p.err != nullptr) atomicOr(p.err, PRCR_DERR_RANGE);
}

}  // namespace

hipError_t launch_reassign(const ReassignParams &p, hipStream_t stream) {
  reassign_kernel<<<dim3(p.batch), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace prcr
