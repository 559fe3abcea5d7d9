// Fused gather -> M-RoPE rebinding -> inject kernel (Eq. (11)-(13)).
//
// One wavefront owns one selected token and a contiguous run of that token's
// (layer, head) rows.  Per token it computes the cos/sin of the token's new
// angles once (one double-precision sincos per lane, then spread to the lanes
// that need it with cross-lane shuffles) and keeps them in registers for every
// row it processes.  Per row, a lane owns one 16-byte chunk of the first half of
// the head dimension and the matching chunk of the second half, so both
// elements of every rotary pair (x_i, x_{i+d/2}) sit in the same lane and no
// data moves between lanes in the hot loop.  K and V rows are read and written
// with 16-byte non-temporal accesses: every byte is touched exactly once.
#include <cmath>

#include "prcr_internal.h"

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

// Compile-time launch shape, chosen by measurement on MI355X: 4 waves per
// workgroup, 2 row iterations in flight per wave, about 72 rows per wave, keys
// and values in separate halves of the grid, non-temporal 16-byte accesses.
#ifndef PRCR_WAVES_PER_BLOCK
#define PRCR_WAVES_PER_BLOCK 4
#endif
#ifndef PRCR_UNROLL
#define PRCR_UNROLL 2
#endif
#ifndef PRCR_ROWS_PER_WAVE
#define PRCR_ROWS_PER_WAVE 72
#endif
#ifndef PRCR_SPLIT_KV
#define PRCR_SPLIT_KV 1
#endif
#ifndef PRCR_NONTEMPORAL
#define PRCR_NONTEMPORAL 1
#endif

__device__ __forceinline__ u32x4 load16(const char *p) {
#if PRCR_NONTEMPORAL
  return load_nt(p);
#else
  return *reinterpret_cast<const u32x4 *>(p);
#endif
}
__device__ __forceinline__ void store16(char *p, u32x4 v) {
#if PRCR_NONTEMPORAL
  store_nt(p, v);
#else
  *reinterpret_cast<u32x4 *>(p) = v;
#endif
}

// One wavefront = one selected token x one run of rows_per_wave (layer, head)
// rows of it.  With kSplitKV the top of the flat workgroup index picks the
// array: the first half rotates and stores keys, the second half copies values.
// Workgroups are dispatched in index order, so the key half runs before the
// value half and each wave streams one source and one destination, which
// measured faster than moving both arrays in one wave.
template <typename T, int D, class Map, bool kPaged, int kWaves, int kUnroll, bool kSplitKV>
__global__ __launch_bounds__(kWaves * kWave) void rebind_inject_kernel(const RebindParams p) {
  constexpr int P = D / 2;
  constexpr int E = Store<T>::kPerChunk;   // elements per 16-byte chunk
  constexpr int LPR = P / E;               // lanes per row
  constexpr int RPI = kWave / LPR;         // rows per wave and iteration
  constexpr int kRowBytes = D * static_cast<int>(sizeof(T));
  constexpr int kHalfBytes = kRowBytes / 2;
  static_assert(Map::kPairs == P, "axis map does not match head_dim");
  static_assert(P % E == 0 && kWave % LPR == 0 && P <= kWave, "unsupported head_dim");

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;

  // Flat workgroup index -> (token block, row group, K|V), token block fastest.
  // Consecutive workgroups (which the dispatcher deals round-robin to the 8 XCDs)
  // take consecutive tokens, so the work in flight spreads over many sequences,
  // memory rows and cache rows at once; orders that concentrate it on fewer
  // sequences, or give each XCD its own contiguous range, measured slower.
  constexpr int nkv = kSplitKV ? 2 : 1;
  const int64_t n_tblk = (static_cast<int64_t>(p.total_k) + kWaves - 1) / kWaves;
  const int64_t n_work = n_tblk * p.n_row_groups * nkv;
  const int64_t L = blockIdx.x;
  // New cache lengths, written once by the first workgroup (also when total_k = 0).
  if (L == 0 && p.new_cache_len != nullptr) {
    for (int b = threadIdx.x; b < p.batch; b += blockDim.x)
      p.new_cache_len[b] = p.cache_len[b] + (p.sel_off[b + 1] - p.sel_off[b]);
  }
  if (L >= n_work) return;
  const int64_t tblk = L % n_tblk;
  const int grp = static_cast<int>((L / n_tblk) % p.n_row_groups);
  const int kv = static_cast<int>(L / (n_tblk * p.n_row_groups));
  const bool keys = !kSplitKV || kv == 0;
  const bool values = !kSplitKV || kv == 1;
  const int g = static_cast<int>(tblk * kWaves + wave);
  if (g >= p.total_k) return;
  const int r = lane / LPR;   // this lane's row within an iteration
  const int c = lane % LPR;   // this lane's 16-byte chunk of a half row

  // Loads that depend only on g are issued first ...
  const int m = p.sel_idx[g];
  double pt = 0.0, ph = 0.0, pw = 0.0;
  if (keys) {
    pt = p.new_pos[3 * static_cast<int64_t>(g) + 0];
    ph = p.new_pos[3 * static_cast<int64_t>(g) + 1];
    pw = p.new_pos[3 * static_cast<int64_t>(g) + 2];
  }
  // ... then the sequence of g: (number of offsets <= g) - 1, by a ballot over
  // the offsets held one per lane ...
  int cnt = 0;
  for (int base = 0; base <= p.batch; base += kWave) {
    const int i = base + lane;
    const bool le = (i <= p.batch) && (p.sel_off[i] <= g);
    cnt += __popcll(__ballot(le));
  }
  const int b = __builtin_amdgcn_readfirstlane(cnt - 1);
  // ... and the per-sequence values, all at once from a clamped index.
  const int bq = min(max(b, 0), p.batch - 1);
  const int s0 = p.sel_off[bq];
  const int s1 = p.sel_off[bq + 1];
  const int nvis = p.n_visual[bq];
  const int64_t slot = static_cast<int64_t>(p.cache_len[bq]) + (g - s0);

  int flags = 0;
  bool ok = b >= 0 && b < p.batch && s0 <= g && g < s1;
  if (!ok) {
    flags = PRCR_DERR_OFFSETS;
  } else if (m < 0 || m >= nvis || m >= p.max_visual) {
    ok = false;
    flags = PRCR_DERR_INDEX;
  }
  int64_t slot_id = -1, blk = 0, off = 0;
  if (ok) {
    if constexpr (kPaged) {
      const int64_t lb = slot >= 0 ? slot / p.block_size : -1;
      if (lb < 0 || lb >= p.max_blocks) {
        ok = false;
        flags = PRCR_DERR_CAPACITY;
      } else {
        blk = p.block_table[static_cast<int64_t>(b) * p.max_blocks + lb];
        if (blk < 0 || blk >= p.n_blocks) {
          ok = false;
          flags = PRCR_DERR_BLOCK;
        } else {
          off = slot - lb * p.block_size;
          slot_id = blk * p.block_size + off;
        }
      }
    } else if (slot < 0 || slot >= p.s_max) {
      ok = false;
      flags = PRCR_DERR_CAPACITY;
    } else {
      slot_id = static_cast<int64_t>(b) * p.s_max + slot;
    }
  }
  if (keys && grp == 0 && lane == 0) {
    if (p.slot_mapping != nullptr) p.slot_mapping[g] = ok ? slot_id : -1;
    if (flags != 0 && p.err != nullptr) atomicOr(p.err, flags);
  }
  if (!ok) return;

  const int rows_total = p.n_layers * p.n_kv_heads;
  const int row0 = grp * p.rows_per_wave;
  const int row_end = min(rows_total, row0 + p.rows_per_wave);
  const size_t tok_off = (static_cast<size_t>(b) * p.max_visual + m) * rows_total;
  // Destination row offsets (in rows of head_dim elements).
  size_t dst_base;
  if constexpr (kPaged) {
    dst_base = static_cast<size_t>(blk) * p.block_size + off;   // slot within a layer's pool
  } else {
    dst_base = static_cast<size_t>(b) * rows_total;             // first (layer, head) row of b
  }
  auto dst_offset = [&](int row) -> size_t {
    if constexpr (kPaged) {
      const int l = row / p.n_kv_heads;
      const int h = row - l * p.n_kv_heads;
      return ((static_cast<size_t>(l) * p.n_blocks * p.block_size + dst_base) * p.n_kv_heads + h) *
             kRowBytes;
    } else {
      return ((dst_base + row) * p.s_max + slot) * kRowBytes;
    }
  };

  if (keys) {
    // cos/sin of this token's angles: lane i computes pair i (mod P), then lane
    // (r, c) gathers the pairs c*E .. c*E+E-1 of its two chunks by shuffles.
    const int pair = lane % P;
    const int ax = Map::axis(pair);
    double sv, cv;
    sincos((ax == 0 ? pt : (ax == 1 ? ph : pw)) * p.inv_freq[pair], &sv, &cv);
    double cs[E], sn[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
      cs[e] = __shfl(cv, c * E + e);
      sn[e] = __shfl(sv, c * E + e);
    }
    const char *src = static_cast<const char *>(p.mem_k) + tok_off * kRowBytes + c * 16;
    char *dst = static_cast<char *>(p.cache_k) + c * 16;
    for (int rb = row0; rb < row_end; rb += RPI * kUnroll) {
      u32x4 lo[kUnroll], hi[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = rb + u * RPI + r;
        if (row < row_end) {
          lo[u] = load16(src + static_cast<size_t>(row) * kRowBytes);
          hi[u] = load16(src + static_cast<size_t>(row) * kRowBytes + kHalfBytes);
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = rb + u * RPI + r;
        if (row < row_end) {
          u32x4 ol, oh;
          Store<T>::rotate(lo[u], hi[u], cs, sn, ol, oh);
          const size_t d = dst_offset(row);
          store16(dst + d, ol);
          store16(dst + d + kHalfBytes, oh);
        }
      }
    }
  }
  if (values) {
    const char *src = static_cast<const char *>(p.mem_v) + tok_off * kRowBytes + c * 16;
    char *dst = static_cast<char *>(p.cache_v) + c * 16;
    for (int rb = row0; rb < row_end; rb += RPI * kUnroll) {
      u32x4 lo[kUnroll], hi[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = rb + u * RPI + r;
        if (row < row_end) {
          lo[u] = load16(src + static_cast<size_t>(row) * kRowBytes);
          hi[u] = load16(src + static_cast<size_t>(row) * kRowBytes + kHalfBytes);
        }
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = rb + u * RPI + r;
        if (row < row_end) {
          const size_t d = dst_offset(row);
          store16(dst + d, lo[u]);
          store16(dst + d + kHalfBytes, hi[u]);
        }
      }
    }
  }
}

constexpr int kWavesPerBlock = PRCR_WAVES_PER_BLOCK;
constexpr int kUnrollRows = PRCR_UNROLL;
constexpr bool kSplit = PRCR_SPLIT_KV != 0;

template <typename T, int D, class Map, bool kPaged>
hipError_t launch_one(const RebindParams &in, hipStream_t stream) {
  constexpr int P = D / 2;
  constexpr int LPR = P / Store<T>::kPerChunk;
  constexpr int RPI = kWave / LPR;
  RebindParams p = in;
  // Rows of one token handled by one wave: a whole number of iterations, about
  // PRCR_ROWS_PER_WAVE, spread evenly over the token's n_layers * n_kv_heads rows.
  const int rows_total = p.n_layers * p.n_kv_heads;
  const int step = RPI * kUnrollRows;
  const int target = (PRCR_ROWS_PER_WAVE + step - 1) / step * step;
  const int groups = (rows_total + target - 1) / target;
  int per = (rows_total + groups - 1) / groups;
  per = (per + step - 1) / step * step;
  p.rows_per_wave = per;
  p.n_row_groups = (rows_total + per - 1) / per;
  if (p.n_row_groups > 65535) return hipErrorInvalidConfiguration;
  // One flat grid over (token block, row group, K|V); at least one workgroup so
  // that the new cache lengths are written when nothing is selected.
  const int64_t n_tblk = (static_cast<int64_t>(p.total_k) + kWavesPerBlock - 1) / kWavesPerBlock;
  int64_t n_work = n_tblk * p.n_row_groups * (kSplit ? 2 : 1);
  if (n_work < 1) n_work = 1;
  if (n_work > INT32_MAX) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<unsigned>(n_work));
  rebind_inject_kernel<T, D, Map, kPaged, kWavesPerBlock, kUnrollRows, kSplit>
      <<<grid, kWavesPerBlock * kWave, 0, stream>>>(p);
  return hipGetLastError();
}

template <typename T, bool kPaged>
hipError_t dispatch_map(const RebindParams &p, int head_dim, AxisMapId map, hipStream_t stream) {
  if (head_dim == 64) {
    if (map == AxisMapId::kS_8_12_12) return launch_one<T, 64, Sectioned<8, 12, 12>, kPaged>(p, stream);
    if (map == AxisMapId::kI_11_11_10) return launch_one<T, 64, Interleaved<11, 11, 10>, kPaged>(p, stream);
  } else if (head_dim == 128) {
    if (map == AxisMapId::kS_16_24_24) return launch_one<T, 128, Sectioned<16, 24, 24>, kPaged>(p, stream);
    if (map == AxisMapId::kI_22_21_21) return launch_one<T, 128, Interleaved<22, 21, 21>, kPaged>(p, stream);
    if (map == AxisMapId::kI_24_20_20) return launch_one<T, 128, Interleaved<24, 20, 20>, kPaged>(p, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

AxisMapId axis_map_id(const prcr_rope &rope) {
  const int *s = rope.section;
  if (rope.head_dim == 64) {
    if (!rope.interleaved && s[0] == 8 && s[1] == 12 && s[2] == 12) return AxisMapId::kS_8_12_12;
    if (rope.interleaved && s[0] == 11 && s[1] == 11 && s[2] == 10) return AxisMapId::kI_11_11_10;
  } else if (rope.head_dim == 128) {
    if (!rope.interleaved && s[0] == 16 && s[1] == 24 && s[2] == 24) return AxisMapId::kS_16_24_24;
    if (rope.interleaved && s[0] == 22 && s[1] == 21 && s[2] == 21) return AxisMapId::kI_22_21_21;
    if (rope.interleaved && s[0] == 24 && s[1] == 20 && s[2] == 20) return AxisMapId::kI_24_20_20;
  }
  return AxisMapId::kUnsupported;
}

int axis_of_pair(AxisMapId id, int i) {
  switch (id) {
    case AxisMapId::kS_8_12_12: return Sectioned<8, 12, 12>::axis(i);
    case AxisMapId::kI_11_11_10: return Interleaved<11, 11, 10>::axis(i);
    case AxisMapId::kS_16_24_24: return Sectioned<16, 24, 24>::axis(i);
    case AxisMapId::kI_22_21_21: return Interleaved<22, 21, 21>::axis(i);
    case AxisMapId::kI_24_20_20: return Interleaved<24, 20, 20>::axis(i);
    default: return -1;
  }
}

hipError_t launch_rebind(const RebindParams &p, prcr_dtype dtype, int head_dim, AxisMapId map,
                         bool paged, hipStream_t stream) {
  if (dtype == PRCR_F32)
    return paged ? dispatch_map<float, true>(p, head_dim, map, stream)
                 : dispatch_map<float, false>(p, head_dim, map, stream);
  return paged ? dispatch_map<uint16_t, true>(p, head_dim, map, stream)
               : dispatch_map<uint16_t, false>(p, head_dim, map, stream);
}

}  // namespace prcr
