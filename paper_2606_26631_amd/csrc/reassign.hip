// Position reassignment for the selected tokens (Sec. 3.2, Eq. (8)-(10)).
//
// One workgroup per sequence: a block-wide min/max over the valid selected
// coordinates (Eq. (8)), then one thread per token writes its new (t, h, w)
// position.  The workgroup has 64-1024 threads, as many as the mean selection
// per sequence needs, so that a typical sequence's tokens are read in one round
// of loads instead of one round per 256 tokens.  PCR positions are the exact rational of Eq. (9)-(10) over integer
// numerator and denominator, divided once in double precision, which makes the
// value the correctly rounded one and identical on every device.
#include <climits>
#include <cmath>

#include "positions.h"
#include "prcr_internal.h"

namespace prcr {
namespace {

__device__ __forceinline__ int wave_min(int v) {
  for (int o = kWave / 2; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_max(int v) {
  for (int o = kWave / 2; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
  return v;
}

template <int kThreads>
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
      bool nb = false;
      p.next_pos[b] = next_pos_int32(p_txt + 1, &nb);
      if (p.err != nullptr) atomicOr(p.err, PRCR_DERR_OFFSETS | (nb ? PRCR_DERR_RANGE : 0));
    }
    // Out-of-range offsets leave this sequence's positions unwritten.
    if (!(s0 >= 0 && s0 <= s1 && s1 <= p.total_k)) return;
  }
  const int K = s1 - s0;
  const int64_t L = p.l_ext;
  // The first selected index of this thread is loaded together with the token
  // count (it does not depend on it).
  const int m_first = tid < K ? p.sel_idx[s0 + tid] : -1;
  const int nvis = min(p.n_visual[b], p.max_visual);
  const int32_t *coords_b = p.coords + static_cast<int64_t>(b) * p.max_visual * 3;

  // Eq. (8): per-axis range over the valid selected tokens.  A thread keeps the
  // index and coordinates of its first token for the second pass (every token,
  // when K <= kThreads), so that pass needs no loads for it.
  int lo[3] = {INT_MAX, INT_MAX, INT_MAX};
  int hi[3] = {INT_MIN, INT_MIN, INT_MIN};
  int bad = 0;
  int c_first[3] = {0, 0, 0};
  for (int j = tid; j < K; j += kThreads) {
    const int m = j == tid ? m_first : p.sel_idx[s0 + j];
    if (m < 0 || m >= nvis) {
      bad = 1;
      continue;
    }
    int cc[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) cc[a] = coords_b[3 * m + a];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      if (j == tid) c_first[a] = cc[a];
      lo[a] = min(lo[a], cc[a]);
      hi[a] = max(hi[a], cc[a]);
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
    const int m = j == tid ? m_first : p.sel_idx[s0 + j];
    double *out = p.new_pos + 3 * static_cast<int64_t>(s0 + j);
    if (m < 0 || m >= nvis) {
      out[0] = out[1] = out[2] = __builtin_nan("");
      continue;
    }
    // All three coordinates are in registers before the first store (the stores
    // could otherwise alias them and force a reload after each one).
    int cc[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) cc[a] = j == tid ? c_first[a] : coords_b[3 * m + a];
    bool rb = false;
    double v[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) v[a] = reassigned(p.mode, p_txt, L, K, j, lo[a], hi[a], cc[a], &rb);
#pragma unroll
    for (int a = 0; a < 3; ++a) out[a] = v[a];
    range_bad |= rb ? 1 : 0;
  }

  if (tid == 0) {
    int64_t span = 0;
    for (int a = 0; a < 3; ++a)
      span = max(span, static_cast<int64_t>(hi[a]) - static_cast<int64_t>(lo[a]));
    const int64_t next = next_text_position(p.mode, p_txt, K, any_valid, span);
    bool nb = false;
    p.next_pos[b] = next_pos_int32(next, &nb);
    if ((bad || nb) && p.err != nullptr)
      atomicOr(p.err, (bad ? PRCR_DERR_INDEX : 0) | (nb ? PRCR_DERR_RANGE : 0));
  }
  if (range_bad && p.err != nullptr) atomicOr(p.err, PRCR_DERR_RANGE);
}

}  // namespace

hipError_t launch_reassign(const ReassignParams &p, hipStream_t stream) {
  const int64_t mean_k = p.batch > 0 ? (static_cast<int64_t>(p.total_k) + p.batch - 1) / p.batch : 0;
  const int threads = mean_k <= 64 ? 64 : (mean_k <= 256 ? 256 : (mean_k <= 512 ? 512 : 1024));
  if (!grid_fits(p.batch, threads)) return hipErrorInvalidConfiguration;
  const dim3 grid(p.batch);
  switch (threads) {
    case 64: reassign_kernel<64><<<grid, dim3(64), 0, stream>>>(p); break;
    case 256: reassign_kernel<256><<<grid, dim3(256), 0, stream>>>(p); break;
    case 512: reassign_kernel<512><<<grid, dim3(512), 0, stream>>>(p); break;
    default: reassign_kernel<1024><<<grid, dim3(1024), 0, stream>>>(p); break;
  }
  return hipGetLastError();
}

}  // namespace prcr
