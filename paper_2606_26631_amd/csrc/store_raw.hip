// Raw Visual Evidence Memory capture (Sec. 3.1, Eq. (6)-(7)).
//
// For one layer, copies the pre-rotary K/V projections of every visual token
// into the token-major memory with 16-byte non-temporal accesses. A wave moves
// one array's rows (keys or values) of kTokens visual tokens of one sequence;
// with a value memory, even workgroups move keys and odd ones values. Waves are
// numbered token-first: consecutive waves take the same tokens of successive
// sequences. A token's row of one layer sits n_layers rows after the previous
// token's, so the stores in flight at one time spread over every sequence's
// memory instead of crowding a few sequences' rows. Over independent
// allocations this order was as fast on average as sequence-first waves, with
// a narrower spread between allocations and a worst case 12 % faster.
#include "prcr_internal.h"

namespace prcr {
namespace {

constexpr int kWaves = 4;
constexpr int kTokens = 2;   // visual tokens per wave
constexpr int kBatch = 2;    // 16-byte chunks per lane and token in one round

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kWaves * kWave) void store_raw_kernel(const StoreParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const bool with_v = p.mem_v != nullptr;   // false for a key-only memory
  const bool values = with_v && (blockIdx.x & 1u) != 0;
  const int64_t wg = with_v ? blockIdx.x >> 1 : blockIdx.x;
  const int64_t w = wg * kWaves + threadIdx.x / kWave;
  const int b = static_cast<int>(w % p.batch);
  const int64_t m0 = w / p.batch * kTokens;
  // The source rows are read together with the count (an entry past the count is
  // in the array and its value unused), so one memory round trip precedes the copy.
  int rows[kTokens];
#pragma unroll
  for (int t = 0; t < kTokens; ++t)
    rows[t] = p.vis_rows[static_cast<int64_t>(b) * p.max_visual + min(m0 + t, static_cast<int64_t>(p.max_visual) - 1)];
  const int n_vis = min(p.n_visual[b], p.max_visual);
  if (m0 >= n_vis) return;
  const char *raw = static_cast<const char *>(values ? p.raw_v : p.raw_k);
  char *mem = static_cast<char *>(values ? p.mem_v : p.mem_k);
  size_t src[kTokens], dst[kTokens];
  bool live[kTokens];
#pragma unroll
  for (int t = 0; t < kTokens; ++t) {
    const int64_t m = m0 + t;
    live[t] = m < n_vis;
    src[t] = dst[t] = 0;
    if (!live[t]) continue;
    const int r = rows[t];
    if (r < 0 || r >= p.s_src) {
      // The key wave of the token reports it; both skip the row.
      if (!values && lane == 0 && p.err != nullptr) atomicOr(p.err, PRCR_DERR_INDEX);
      live[t] = false;
      continue;
    }
    src[t] = (static_cast<size_t>(b) * p.s_src + r) * p.row_bytes;
    dst[t] = ((static_cast<size_t>(b) * p.max_visual + m) * p.n_layers + p.layer) * p.row_bytes;
  }
  // Every load of a round (up to kBatch chunks of each token per lane) is issued
  // before its stores.
  for (int64_t o0 = lane * 16; o0 < p.row_bytes; o0 += kWave * 16 * kBatch) {
    u32x4 x[kTokens][kBatch];
#pragma unroll
    for (int t = 0; t < kTokens; ++t) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int64_t o = o0 + u * kWave * 16;
        if (live[t] && o < p.row_bytes)
          x[t][u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(raw + src[t] + o));
      }
    }
#pragma unroll
    for (int t = 0; t < kTokens; ++t) {
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const int64_t o = o0 + u * kWave * 16;
        if (live[t] && o < p.row_bytes)
          __builtin_nontemporal_store(x[t][u], reinterpret_cast<u32x4 *>(mem + dst[t] + o));
      }
    }
  }
}

}  // namespace

hipError_t launch_store(const StoreParams &p, hipStream_t stream) {
  const int64_t waves = (static_cast<int64_t>(p.max_visual) + kTokens - 1) / kTokens * p.batch;
  const int64_t blocks = (waves + kWaves - 1) / kWaves * (p.mem_v != nullptr ? 2 : 1);
  if (!grid_fits(blocks, kWaves * kWave)) return hipErrorInvalidConfiguration;
  store_raw_kernel<<<static_cast<unsigned>(blocks), kWaves * kWave, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace prcr
