// Reference copy kernels for the bandwidth measurement (not part of the PRCR
// path): what a plain device copy attains on this GPU, and what a copy with
// exactly the rebinding kernel's addresses attains.
//
//   prcr_copyref_stream   src -> dst, each workgroup owning one contiguous chunk:
//                         the attainable read + write rate of the GPU.
//   prcr_copyref_pattern  the rebind's own access pattern with no arithmetic and no
//                         metadata: per selected token, its (layer, head) rows are
//                         read from one contiguous run of the memory and written to
//                         the cache rows of its slot, with the rebinding kernel's
//                         wave structure (one wave per token x run of rows, four
//                         waves per workgroup, 16-row load batches with the next
//                         batch in flight) and dispatch order (token fastest, then
//                         row group, then the key array before the value array).
//
// Both use 16-byte non-temporal loads and stores, as the rebind does.  Offsets
// are byte offsets computed by the caller, who checks them against the arrays.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld(const char *p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
}
__device__ __forceinline__ void st(char *p, u32x4 v) {
  __builtin_nontemporal_store(v, reinterpret_cast<u32x4 *>(p));
}

constexpr int kThreads = 256;
constexpr int kStreamUnroll = 4;     // 16-byte chunks per thread per pass: 16 KB per workgroup

__global__ __launch_bounds__(kThreads) void stream_kernel(const char *src, char *dst, int64_t bytes,
                                                          int64_t chunk) {
  const int64_t base = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t end = base + chunk < bytes ? base + chunk : bytes;
  for (int64_t i = base + threadIdx.x * 16; i < end; i += kStreamUnroll * kThreads * 16) {
    u32x4 v[kStreamUnroll];
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) {
      const int64_t j = i + static_cast<int64_t>(u) * kThreads * 16;
      if (j < end) v[u] = ld(src + j);
    }
#pragma unroll
    for (int u = 0; u < kStreamUnroll; ++u) {
      const int64_t j = i + static_cast<int64_t>(u) * kThreads * 16;
      if (j < end) st(dst + j, v[u]);
    }
  }
}

struct PatternParams {
  const char *src[2];          // key memory, value memory
  char *dst[2];                // key cache, value cache
  const int64_t *src_tok;      // [n_tok] byte offset of token g's first row in the memory
  const int64_t *dst_tok;      // [n_tok] byte offset of token g's row 0 in the cache
  int64_t group_stride;        // cache byte distance between consecutive row groups of G rows
  int32_t n_tok, rows_total, rows_per_wave, n_row_groups, group_log2;
};

// Row r of a token goes from src_tok + r * 256 to
// dst_tok + (r >> group_log2) * group_stride + (r & (2^group_log2 - 1)) * 256:
// contiguous caches use group_log2 = 0 and the cache's row stride, paged caches
// the KV-head count and the layer stride of the block pool.  Rows are 256 bytes
// (head_dim 128, bf16).  As in the rebinding kernel, a lane holds one 16-byte
// chunk of the first half of a row and the same chunk of the second half (8
// lanes per row, 8 rows per pass), two passes per batch of loads.
__global__ __launch_bounds__(kThreads) void pattern_kernel(const PatternParams p) {
  constexpr int kRowBytes = 256, kHalf = 128, kLanesPerRow = 8, kRowsPerPass = 8, kUnroll = 2;
  constexpr int kStep = kRowsPerPass * kUnroll;        // 16 rows per batch of loads
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t n_tblk = (static_cast<int64_t>(p.n_tok) + 3) / 4;
  const int64_t L = blockIdx.x;
  const int64_t tblk = L % n_tblk;
  const int grp = static_cast<int>((L / n_tblk) % p.n_row_groups);
  const int arr = L < n_tblk * p.n_row_groups ? 0 : 1;
  const int64_t g = tblk * 4 + wave;
  if (g >= p.n_tok) return;
  const int r = lane / kLanesPerRow, c = lane % kLanesPerRow;
  const int row0 = grp * p.rows_per_wave;
  const int row_end = min(p.rows_total, row0 + p.rows_per_wave);
  const int gmask = (1 << p.group_log2) - 1;
  const char *s = p.src[arr] + p.src_tok[g] + c * 16;
  char *d = p.dst[arr] + p.dst_tok[g] + c * 16;
  auto dst_off = [&](int row) -> int64_t {
    return static_cast<int64_t>(row >> p.group_log2) * p.group_stride +
           static_cast<int64_t>(row & gmask) * kRowBytes;
  };
  u32x4 lo[kUnroll], hi[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int64_t o = static_cast<int64_t>(min(row0 + u * kRowsPerPass + r, row_end - 1)) * kRowBytes;
    lo[u] = ld(s + o);
    hi[u] = ld(s + o + kHalf);
  }
  int rb = row0;
  for (; rb + kStep < row_end; rb += kStep) {
    u32x4 nlo[kUnroll], nhi[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t o =
          static_cast<int64_t>(min(rb + kStep + u * kRowsPerPass + r, row_end - 1)) * kRowBytes;
      nlo[u] = ld(s + o);
      nhi[u] = ld(s + o + kHalf);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t o = dst_off(rb + u * kRowsPerPass + r);
      st(d + o, lo[u]);
      st(d + o + kHalf, hi[u]);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      lo[u] = nlo[u];
      hi[u] = nhi[u];
    }
  }
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const int row = rb + u * kRowsPerPass + r;
    if (row < row_end) {
      const int64_t o = dst_off(row);
      st(d + o, lo[u]);
      st(d + o + kHalf, hi[u]);
    }
  }
}

}  // namespace

extern "C" {

// Copies `bytes` (a multiple of 16) from src to dst, `chunk` bytes per workgroup.
int prcr_copyref_stream(const void *src, void *dst, int64_t bytes, int64_t chunk,
                        hipStream_t stream) {
  if (src == nullptr || dst == nullptr || bytes <= 0 || bytes % 16 != 0 || chunk <= 0 ||
      chunk % 16 != 0)
    return 1;
  const int64_t grid = (bytes + chunk - 1) / chunk;
  if (grid > 0x7FFFFFFF / kThreads) return 2;
  stream_kernel<<<dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, stream>>>(
      static_cast<const char *>(src), static_cast<char *>(dst), bytes, chunk);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

// The rebind's access pattern over two arrays (keys, then values); see above.
int prcr_copyref_pattern(const void *src_k, const void *src_v, void *dst_k, void *dst_v,
                         const int64_t *src_tok, const int64_t *dst_tok, int32_t n_tok,
                         int32_t rows_total, int32_t rows_per_wave, int32_t group_log2,
                         int64_t group_stride, hipStream_t stream) {
  if (src_k == nullptr || src_v == nullptr || dst_k == nullptr || dst_v == nullptr ||
      src_tok == nullptr || dst_tok == nullptr || n_tok < 1 || rows_total < 1 ||
      rows_per_wave < 1 || group_log2 < 0 || group_log2 > 8)
    return 1;
  PatternParams p{};
  p.src[0] = static_cast<const char *>(src_k);
  p.src[1] = static_cast<const char *>(src_v);
  p.dst[0] = static_cast<char *>(dst_k);
  p.dst[1] = static_cast<char *>(dst_v);
  p.src_tok = src_tok;
  p.dst_tok = dst_tok;
  p.group_stride = group_stride;
  p.n_tok = n_tok;
  p.rows_total = rows_total;
  p.rows_per_wave = rows_per_wave;
  p.n_row_groups = (rows_total + rows_per_wave - 1) / rows_per_wave;
  p.group_log2 = group_log2;
  const int64_t grid = (static_cast<int64_t>(n_tok) + 3) / 4 * p.n_row_groups * 2;
  if (grid > 0x7FFFFFFF / kThreads) return 2;
  pattern_kernel<<<dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
