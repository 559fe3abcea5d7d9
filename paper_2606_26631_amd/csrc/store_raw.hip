// Raw Visual Evidence Memory capture (Sec. 3.1, Eq. (6)-(7)).
//
// For one layer, copies the pre-rotary K/V projections of every visual token
// into the token-major memory: one wavefront per (sequence, visual token) moves
// the token's n_kv_heads * head_dim row with 16-byte accesses.
#include "prcr_internal.h"

namespace prcr {
namespace {

constexpr int kWaves = 4;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kWaves * kWave) void store_raw_kernel(const StoreParams p) {
  const int lane = threadIdx.x & (kWave - 1);
  const int m = blockIdx.x * kWaves + threadIdx.x / kWave;
  const int b = blockIdx.y;
  if (m >= p.max_visual || m >= p.n_visual[b]) return;
  const int r = p.vis_rows[static_cast<int64_t>(b) * p.max_visual + m];
  if (r < 0 || r >= p.s_src) {
    if (lane == 0 && p.err != nullptr) atomicOr(p.err, PRCR_DERR_INDEX);
    return;
  }
  const size_t src = (static_cast<size_t>(b) * p.s_src + r) * p.row_bytes;
  const size_t dst = ((static_cast<size_t>(b) * p.max_visual + m) * p.n_layers + p.layer) * p.row_bytes;
  const char *sk = static_cast<const char *>(p.raw_k) + src;
  char *dk = static_cast<char *>(p.mem_k) + dst;
  const bool with_v = p.mem_v != nullptr;   // false for a key-only memory
  const char *sv = with_v ? static_cast<const char *>(p.raw_v) + src : nullptr;
  char *dv = with_v ? static_cast<char *>(p.mem_v) + dst : nullptr;
  // Up to kBatch 16-byte chunks of each array per lane in flight: every load of
  // the batch is issued before its stores.
  constexpr int kBatch = 2;
  for (int o0 = lane * 16; o0 < p.row_bytes; o0 += kWave * 16 * kBatch) {
    u32x4 k[kBatch], v[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int o = o0 + u * kWave * 16;
      if (o < p.row_bytes) {
        k[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(sk + o));
        if (with_v) v[u] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(sv + o));
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int o = o0 + u * kWave * 16;
      if (o < p.row_bytes) {
        __builtin_nontemporal_store(k[u], reinterpret_cast<u32x4 *>(dk + o));
        if (with_v) __builtin_nontemporal_store(v[u], reinterpret_cast<u32x4 *>(dv + o));
      }
    }
  }
}

}  // namespace

hipError_t launch_store(const StoreParams &p, hipStream_t stream) {
  const int64_t blocks = (static_cast<int64_t>(p.max_visual) + kWaves - 1) / kWaves;
  if (!grid_fits(blocks, kWaves * kWave)) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<unsigned>(blocks), p.batch);
  store_raw_kernel<<<grid, kWaves * kWave, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace prcr
