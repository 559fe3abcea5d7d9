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

template <typename T, int D, class Map, bool kPaged, int kWaves, int kUnroll>
__global__ __launch_bounds__(kWaves * kWave) void rebind_inject_kernel(const RebindParams p) {
  constexpr int P = D / 2;
  constexpr int E = Store<T>::kPerChunk;   // elements per 16-byte chunk
  constexpr int LPR = P / E;               // lanes per row
  constexpr int RPI = kWave / LPR;         // rows per wave per iteration
  constexpr int kRowBytes = D * static_cast<int>(sizeof(T));
  constexpr int kHalfBytes = kRowBytes / 2;
  static_assert(Map::kPairs == P, "axis map does not match head_dim");
  static_assert(P % E == 0 && kWave % LPR == 0 && P <= kWave, "unsupported head_dim");

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;

  // New cache lengths, written once by the first workgroup (also when total_k = 0).
  if (blockIdx.x == 0 && blockIdx.y == 0 && p.new_cache_len != nullptr) {
    for (int b = threadIdx.x; b < p.batch; b += blockDim.x)
      p.new_cache_len[b] = p.cache_len[b] + (p.sel_off[b + 1] - p.sel_off[b]);
  }

  const int g = blockIdx.x * kWaves + wave;
  if (g >= p.total_k) return;
  const int grp = blockIdx.y;

  // Sequence of token g: (number of offsets <= g) - 1.
  int cnt = 0;
  for (int base = 0; base <= p.batch; base += kWave) {
    const int i = base + lane;
    const bool le = (i <= p.batch) && (p.sel_off[i] <= g);
    cnt += __popcll(__ballot(le));
  }
  const int b = __builtin_amdgcn_readfirstlane(cnt - 1);

  // Per-token validation; every lane sees the same values.
  int flags = 0;
  int m = -1, slot = 0;
  int64_t slot_id = -1;
  int blk = 0, off = 0;
  bool ok = b >= 0 && b < p.batch;
  int s0 = 0;
  if (ok) {
    s0 = p.sel_off[b];
    ok = s0 <= g && g < p.sel_off[b + 1];
  }
  if (!ok) {
    flags = PRCR_DERR_OFFSETS;
  } else {
    m = p.sel_idx[g];
    if (m < 0 || m >= p.n_visual[b] || m >= p.max_visual) {
      ok = false;
      flags = PRCR_DERR_INDEX;
    } else {
      const int64_t slot64 = static_cast<int64_t>(p.cache_len[b]) + (g - s0);
      slot = static_cast<int>(slot64);
      if constexpr (kPaged) {
        const int64_t lb = slot64 >= 0 ? slot64 / p.block_size : -1;
        if (lb < 0 || lb >= p.max_blocks) {
          ok = false;
          flags = PRCR_DERR_CAPACITY;
        } else {
          blk = p.block_table[static_cast<int64_t>(b) * p.max_blocks + lb];
          if (blk < 0 || blk >= p.n_blocks) {
            ok = false;
            flags = PRCR_DERR_BLOCK;
          } else {
            off = static_cast<int>(slot64 - lb * p.block_size);
            slot_id = static_cast<int64_t>(blk) * p.block_size + off;
          }
        }
      } else {
        if (slot64 < 0 || slot64 >= p.s_max) {
          ok = false;
          flags = PRCR_DERR_CAPACITY;
        } else {
          slot_id = static_cast<int64_t>(b) * p.s_max + slot;
        }
      }
    }
  }
  if (grp == 0 && lane == 0) {
    if (p.slot_mapping != nullptr) p.slot_mapping[g] = ok ? slot_id : -1;
    if (flags != 0 && p.err != nullptr) atomicOr(p.err, flags);
  }
  if (!ok) return;

  // cos/sin of this token's angles: lane i computes pair i (mod P) ...
  const double pt = p.new_pos[3 * static_cast<int64_t>(g) + 0];
  const double ph = p.new_pos[3 * static_cast<int64_t>(g) + 1];
  const double pw = p.new_pos[3 * static_cast<int64_t>(g) + 2];
  const int pair = lane % P;
  const int ax = Map::axis(pair);
  const double pos = ax == 0 ? pt : (ax == 1 ? ph : pw);
  double sv, cv;
  sincos(pos * p.inv_freq[pair], &sv, &cv);
  // ... and lane (r, c) gathers the pairs c*E .. c*E+E-1 of its two chunks.
  const int r = lane / LPR;
  const int c = lane % LPR;
  double cs[E], sn[E];
#pragma unroll
  for (int e = 0; e < E; ++e) {
    cs[e] = __shfl(cv, c * E + e);
    sn[e] = __shfl(sv, c * E + e);
  }

  const int rows_total = p.n_layers * p.n_kv_heads;
  const int row0 = grp * p.rows_per_wave;
  const int row_end = min(rows_total, row0 + p.rows_per_wave);
  const size_t tok_off = (static_cast<size_t>(b) * p.max_visual + m) * rows_total;
  const char *src_k = static_cast<const char *>(p.mem_k) + tok_off * kRowBytes + c * 16;
  const char *src_v = static_cast<const char *>(p.mem_v) + tok_off * kRowBytes + c * 16;
  char *dst_k = static_cast<char *>(p.cache_k) + c * 16;
  char *dst_v = static_cast<char *>(p.cache_v) + c * 16;
  // Destination row offset (in rows of D elements) for row index `row` of the token.
  size_t dst_base;
  if constexpr (kPaged) {
    dst_base = static_cast<size_t>(blk) * p.block_size + off;   // slot within a layer's pool
  } else {
    dst_base = static_cast<size_t>(b) * rows_total;             // first (layer, head) row of b
  }

  for (int rb = row0; rb < row_end; rb += RPI * kUnroll) {
    u32x4 kl[kUnroll], kh[kUnroll], vl[kUnroll], vh[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int row = rb + u * RPI + r;
      if (row < row_end) {
        const size_t o = static_cast<size_t>(row) * kRowBytes;
        kl[u] = load_nt(src_k + o);
        kh[u] = load_nt(src_k + o + kHalfBytes);
        vl[u] = load_nt(src_v + o);
        vh[u] = load_nt(src_v + o + kHalfBytes);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int row = rb + u * RPI + r;
      if (row < row_end) {
        size_t d;
        if constexpr (kPaged) {
          const int l = row / p.n_kv_heads;
          const int h = row - l * p.n_kv_heads;
          d = ((static_cast<size_t>(l) * p.n_blocks * p.block_size + dst_base) * p.n_kv_heads + h) *
              kRowBytes;
        } else {
          d = ((dst_base + row) * p.s_max + slot) * kRowBytes;
        }
        u32x4 ol, oh;
        Store<T>::rotate(kl[u], kh[u], cs, sn, ol, oh);
        store_nt(dst_k + d, ol);
        store_nt(dst_k + d + kHalfBytes, oh);
        store_nt(dst_v + d, vl[u]);
        store_nt(dst_v + d + kHalfBytes, vh[u]);
      }
    }
  }
}

constexpr int kWavesPerBlock = 4;
constexpr int kUnrollRows = 2;

template <typename T, int D, class Map, bool kPaged>
hipError_t launch_one(const RebindParams &p, hipStream_t stream) {
  const int bx = p.total_k > 0 ? (p.total_k + kWavesPerBlock - 1) / kWavesPerBlock : 1;
  const dim3 grid(bx, p.n_row_groups > 0 ? p.n_row_groups : 1);
  rebind_inject_kernel<T, D, Map, kPaged, kWavesPerBlock, kUnrollRows>
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
