// Reference copy kernels for the bandwidth measurement (not part of the PRCR
// path): what a plain device copy attains on this GPU, and what a copy with
// exactly the rebinding kernel's addresses attains.
//
//   prcr_copyref_stream   src -> dst, each workgroup owning one contiguous chunk:
//                         the attainable read + write rate of the GPU.
//   prcr_copyref_decode_read  decode attention's reads with no arithmetic: every K and
//                         V row of one layer's attended slots, with the bf16
//                         decode kernel's split of each sequence over workgroups,
//                         tiles, lane layouts and loads in flight.
//   prcr_copyref_prefill  prefill capture's access pattern with no arithmetic: one
//                         layer's raw K/V rows of every prompt token to the
//                         contiguous cache at slot s, and visual tokens' rows to the
//                         memory, with the prefill kernel's wave mapping (8
//                         consecutive (token, head) rows per wave, lane layout as
//                         in the rebind).
//   prcr_copyref_pattern  the rebind's own access pattern with no arithmetic and no
//                         metadata: per selected token, its (layer, head) rows are
//                         read from one contiguous run of the memory and written to
//                         the cache rows of its slot, with the rebinding kernel's
//                         wave structure (one wave per token x run of rows, four
//                         waves per workgroup, 16-row load batches with the next
//                         batch in flight) and dispatch order (token fastest, then
//                         row group, then the key array before the value array).
//
// They use 16-byte non-temporal loads and stores, as the rebind does (the decode
// read's key loads are plain, as in the decode kernel).  Offsets
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

struct DecodeReadParams {
  const char *k;               // cache keys
  const char *v;               // cache values
  const int32_t *block_table;  // paged: [batch][max_blocks]
  const int32_t *len;          // [batch] attended slots
  uint32_t *out;               // [gridDim.z][gridDim.y][gridDim.x] one word per workgroup
  int32_t n_layers, n_kv_heads, layer, s_max, block_size, max_blocks, n_blocks, n_split, paged;
};

// One workgroup per (split, KV head, sequence), as the decode kernel launches them
// (sequences taken longest first), with the bf16 decode kernel's accesses.  Rows are 256 bytes (head_dim 128, bf16).
// The sequence's keys are split in whole rounds of 64 keys; a wave takes tiles of
// 16 keys 64 keys apart.  Key rows are read in the matrix-product operand layout
// (lane l: row l % 16, 16-byte chunks l / 16 + 4 * kk, plain loads), value rows 16
// lanes to a row (non-temporal loads); one buffer of each, the next tile's keys
// loaded once this tile's keys are used and its values once this tile's values
// are.  Paged caches whose blocks are whole tiles take one block-table entry per
// tile from a per-wave register filled 64 tiles at a time; others read an entry
// per key.  Keys past the chunk (or in a block outside the pool) read the head's
// first row, as in the decode kernel.  The words read are folded into one value
// per workgroup so that the loads are kept.
template <bool kPaged, bool kTileBlocks>
__global__ __launch_bounds__(kThreads) void decode_read_kernel(const DecodeReadParams p) {
  constexpr int kRowBytes = 256, kTile = 16, KPB = 64, KK = 4, VL = 4, KPW = 4;
  const int split = blockIdx.x, kvh = blockIdx.y;
  const int lane = threadIdx.x & 63;
  // Rows of workgroups go to the sequences longest first, as in the decode kernel.
  int b = blockIdx.z;
  if (gridDim.z <= 64) {
    const int nb = static_cast<int>(gridDim.z);
    const int mine = lane < nb ? max(p.len[lane], 0) : -1;
    int rank = 0;
    for (int i = 0; i < nb; ++i) {
      const int other = __builtin_amdgcn_readlane(mine, i);
      rank += (other > mine) || (other == mine && i < lane);
    }
    const unsigned long long hit = __ballot(lane < nb && rank == static_cast<int>(blockIdx.z));
    b = hit ? __ffsll(static_cast<long long>(hit)) - 1 : b;
  }
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kt = lane % kTile, kj = lane / kTile;
  const int vr = lane / 16, vc = lane % 16;
  // lengths clamped to the capacity, and block-table entries outside the pool
  // read the head's first row instead, as in the decode kernel: every access stays
  // inside the arrays whatever the inputs
  const int64_t cap = kPaged ? static_cast<int64_t>(p.max_blocks) * p.block_size : p.s_max;
  const int len = static_cast<int>(min(max(static_cast<int64_t>(p.len[b]), int64_t{0}), cap));
  const int per = (len + p.n_split - 1) / p.n_split;
  const int chunk = (per + KPB - 1) / KPB * KPB;
  const int j0 = min(len, split * chunk), j1 = min(len, j0 + chunk);
  const int64_t row_base =
      kPaged ? 0 : ((static_cast<int64_t>(b) * p.n_layers + p.layer) * p.n_kv_heads + kvh) * p.s_max;
  const int64_t row_any =
      kPaged ? static_cast<int64_t>(p.layer) * p.n_blocks * p.block_size * p.n_kv_heads + kvh : row_base;
  auto table = [&](int j) -> int32_t {
    const int js = j < j1 ? j : 0;
    return p.block_table[static_cast<int64_t>(b) * p.max_blocks + js / p.block_size];
  };
  // Rows selected without branches, as in the decode kernel.
  auto row_of = [&](int tb, int j, int lim, int32_t tile_blk) -> int64_t {
    if constexpr (!kPaged) {
      return j < lim ? row_base + j : row_any;
    } else {
      const int32_t blk = kTileBlocks ? tile_blk : table(j);
      const int off = kTileBlocks ? (tb % p.block_size) + (j - tb) : j % p.block_size;
      const int64_t row =
          ((static_cast<int64_t>(p.layer) * p.n_blocks + blk) * p.block_size + off) * p.n_kv_heads + kvh;
      return j < lim && blk >= 0 && blk < p.n_blocks ? row : row_any;
    }
  };
  uint32_t acc = 0;
  const int jw = j0 + wave * kTile;
  const int n_tiles = jw < j1 ? (j1 - jw + KPB - 1) / KPB : 0;
  const int rounds = kTileBlocks ? (n_tiles + 63) / 64 : (n_tiles > 0 ? 1 : 0);
  for (int r = 0; r < rounds; ++r) {
    const int n0 = r * 64;
    int32_t tab = 0;
    if constexpr (kTileBlocks) tab = table(jw + (n0 + lane) * KPB);
    const int lim = kTileBlocks ? static_cast<int>(min(static_cast<int64_t>(j1),
                                                       static_cast<int64_t>(jw) + static_cast<int64_t>(n0 + 64) * KPB))
                                : j1;
    auto blk_of = [&](int n) -> int32_t {
      if constexpr (kTileBlocks) return __builtin_amdgcn_readlane(tab, min(n - n0, 63));
      return 0;
    };
    auto load_k = [&](int tb, int32_t blk, u32x4 *kd) {
      const char *kp = p.k + row_of(tb, tb + kt, lim, blk) * kRowBytes + kj * 16;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) kd[kk] = *reinterpret_cast<const u32x4 *>(kp + kk * 64);
    };
    auto load_v = [&](int tb, int32_t blk, u32x4 *vd) {
#pragma unroll
      for (int u = 0; u < VL; ++u) vd[u] = ld(p.v + row_of(tb, tb + KPW * u + vr, lim, blk) * kRowBytes + vc * 16);
    };
    u32x4 kr[KK], vv[VL];
    int n = n0, jt = jw + n0 * KPB;
    int32_t blk = blk_of(n);
    load_k(jt, blk, kr);
    load_v(jt, blk, vv);
    while (jt < lim) {
      const int32_t blk_n = blk_of(n + 1);
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) acc ^= kr[kk].x ^ kr[kk].y ^ kr[kk].z ^ kr[kk].w;
      load_k(jt + KPB, blk_n, kr);
#pragma unroll
      for (int u = 0; u < VL; ++u) acc ^= vv[u].x ^ vv[u].y ^ vv[u].z ^ vv[u].w;
      load_v(jt + KPB, blk_n, vv);
      jt += KPB;
      ++n;
    }
  }
  for (int o = 32; o > 0; o >>= 1) acc ^= __shfl_xor(acc, o);
  __shared__ uint32_t s_acc[kThreads / 64];
  if (lane == 0) s_acc[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t a = 0;
    for (int w = 0; w < kThreads / 64; ++w) a ^= s_acc[w];
    p.out[(static_cast<int64_t>(b) * gridDim.y + kvh) * gridDim.x + split] = a;
  }
}

struct PrefillPatternParams {
  const char *raw_k, *raw_v;   // [batch][s_src][H][128] bf16 rows
  const int32_t *vis_index;    // [batch][s_src]: visual index or -1
  const int32_t *n_tokens;     // [batch]
  char *cache_k, *cache_v;     // contiguous [batch][n_layers][H][s_max][128]
  char *mem_k, *mem_v;         // [batch][max_visual][n_layers][H][128]
  int32_t batch, s_src, n_kv_heads, n_layers, layer, s_max, max_visual;
};

// Rows are 256 bytes (head_dim 128, bf16); row R = (b * s_src + s) * H + h.
__global__ __launch_bounds__(kThreads) void prefill_pattern_kernel(const PrefillPatternParams p) {
  constexpr int kRowBytes = 256, kHalf = 128, kLanesPerRow = 8, kRowsPerWave = 8;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int H = p.n_kv_heads;
  const int64_t rows_all = static_cast<int64_t>(p.batch) * p.s_src * H;
  const int64_t R = (static_cast<int64_t>(blockIdx.x) * 4 + wave) * kRowsPerWave + lane / kLanesPerRow;
  if (R >= rows_all) return;
  const int c = lane % kLanesPerRow;
  const int b = static_cast<int>(R / (static_cast<int64_t>(p.s_src) * H));
  const int64_t rem = R - static_cast<int64_t>(b) * p.s_src * H;
  const int s = static_cast<int>(rem / H), h = static_cast<int>(rem - static_cast<int64_t>(s) * H);
  const int nt = p.n_tokens[b];
  const int m = p.vis_index[static_cast<int64_t>(b) * p.s_src + s];
  if (s >= nt || s >= p.s_max) return;
  const int64_t o = R * kRowBytes + c * 16;
  const u32x4 kl = ld(p.raw_k + o), kh = ld(p.raw_k + o + kHalf);
  const u32x4 vl = ld(p.raw_v + o), vh = ld(p.raw_v + o + kHalf);
  const int64_t d = ((((static_cast<int64_t>(b) * p.n_layers + p.layer) * H + h) * p.s_max) + s) * kRowBytes + c * 16;
  st(p.cache_k + d, kl);
  st(p.cache_k + d + kHalf, kh);
  st(p.cache_v + d, vl);
  st(p.cache_v + d + kHalf, vh);
  if (m >= 0 && m < p.max_visual) {
    const int64_t mo = (((static_cast<int64_t>(b) * p.max_visual + m) * p.n_layers + p.layer) * H + h) * kRowBytes +
                       c * 16;
    st(p.mem_k + mo, kl);
    st(p.mem_k + mo + kHalf, kh);
    st(p.mem_v + mo, vl);
    st(p.mem_v + mo + kHalf, vh);
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

// Decode attention's reads of one layer (see above): n_split workgroups per
// (sequence, KV head); out holds batch * n_kv_heads * n_split words.
int prcr_copyref_decode_read(const void *k, const void *v, const int32_t *block_table,
                             const int32_t *len, uint32_t *out, int32_t batch, int32_t n_layers,
                             int32_t n_kv_heads, int32_t layer, int32_t s_max, int32_t block_size,
                             int32_t max_blocks, int32_t n_blocks, int32_t n_split, int32_t paged,
                             hipStream_t stream) {
  if (k == nullptr || v == nullptr || len == nullptr || out == nullptr || batch < 1 ||
      batch > 65535 || n_kv_heads < 1 || n_kv_heads > 65535 || n_split < 1 || layer < 0 ||
      layer >= n_layers || (paged && (block_table == nullptr || block_size < 1 || max_blocks < 1 ||
                                      n_blocks < 1)) || (!paged && s_max < 1))
    return 1;
  DecodeReadParams p{};
  p.k = static_cast<const char *>(k);
  p.v = static_cast<const char *>(v);
  p.block_table = block_table;
  p.len = len;
  p.out = out;
  p.n_layers = n_layers;
  p.n_kv_heads = n_kv_heads;
  p.layer = layer;
  p.s_max = s_max;
  p.block_size = block_size;
  p.max_blocks = max_blocks;
  p.n_blocks = n_blocks;
  p.n_split = n_split;
  p.paged = paged;
  const dim3 grid(n_split, n_kv_heads, batch);
  if (!paged)
    decode_read_kernel<false, false><<<grid, dim3(kThreads), 0, stream>>>(p);
  else if (block_size % 16 == 0)
    decode_read_kernel<true, true><<<grid, dim3(kThreads), 0, stream>>>(p);
  else
    decode_read_kernel<true, false><<<grid, dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

// Prefill capture's access pattern for one layer (see above).
int prcr_copyref_prefill(const void *raw_k, const void *raw_v, const int32_t *vis_index,
                         const int32_t *n_tokens, void *cache_k, void *cache_v, void *mem_k,
                         void *mem_v, int32_t batch, int32_t s_src, int32_t n_kv_heads,
                         int32_t n_layers, int32_t layer, int32_t s_max, int32_t max_visual,
                         hipStream_t stream) {
  if (raw_k == nullptr || raw_v == nullptr || vis_index == nullptr || n_tokens == nullptr ||
      cache_k == nullptr || cache_v == nullptr || mem_k == nullptr || mem_v == nullptr ||
      batch < 1 || s_src < 1 || n_kv_heads < 1 || layer < 0 || layer >= n_layers || s_max < 1 ||
      max_visual < 1)
    return 1;
  PrefillPatternParams p{};
  p.raw_k = static_cast<const char *>(raw_k);
  p.raw_v = static_cast<const char *>(raw_v);
  p.vis_index = vis_index;
  p.n_tokens = n_tokens;
  p.cache_k = static_cast<char *>(cache_k);
  p.cache_v = static_cast<char *>(cache_v);
  p.mem_k = static_cast<char *>(mem_k);
  p.mem_v = static_cast<char *>(mem_v);
  p.batch = batch;
  p.s_src = s_src;
  p.n_kv_heads = n_kv_heads;
  p.n_layers = n_layers;
  p.layer = layer;
  p.s_max = s_max;
  p.max_visual = max_visual;
  const int64_t rows = static_cast<int64_t>(batch) * s_src * n_kv_heads;
  const int64_t grid = (rows + 31) / 32;
  if (grid > 0x7FFFFFFF / kThreads) return 2;
  prefill_pattern_kernel<<<dim3(static_cast<unsigned>(grid)), dim3(kThreads), 0, stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
