// Decode attention over the active cache (Eq. (14)): for each sequence and query
// head, softmax(RoPE(q, p_next) K^T * scale) V over the cache_len[b] keys of one
// layer, with grouped-query attention (n_q_heads = G * n_kv_heads, query head
// qh reads KV head qh / G).  The query is a text token, so its three M-RoPE
// positions are equal and the rotation is the 1-D one at p_next.
//
// Split-K flash decoding.  Kernel 1: one workgroup per (key chunk, KV head,
// sequence) streams its keys and values once for all G query heads of the
// group, and the sequence's keys are split evenly over its workgroups, about as
// many workgroups in all as the chip holds at once (with at most 64 sequences,
// the grid's sequence rows take the sequences longest first).  bf16 caches take the
// scores of 16 keys at a time from matrix-core products (decode_partial_bf16_kernel);
// float32 caches take a 16-byte chunk of a key row per lane with scores reduced
// across the lanes of a row by DPP lane permutations (decode_partial_kernel).
// Both keep an online softmax in float32 that rescales only when a running
// maximum rose.  The workgroup's waves are merged in LDS and one (max, sum,
// weighted V) partial per query head and chunk is written to the caller's
// workspace.  Kernel 2 merges the chunks.
#include <cfloat>
#include <climits>
#include <cmath>
#include <type_traits>

#include "prcr_internal.h"
#include "rotary.h"

namespace prcr {
namespace {

#ifndef PRCR_DEC_ITERS
#define PRCR_DEC_ITERS 2
#endif
#ifndef PRCR_DEC_WORKGROUPS
#define PRCR_DEC_WORKGROUPS 0    // workgroups per call; 0: as many as are resident at once
#endif
#ifndef PRCR_DEC_MFMA
#define PRCR_DEC_MFMA 1
#endif
#ifndef PRCR_DEC_WAVES
#define PRCR_DEC_WAVES 4
#endif
constexpr int kWaves = PRCR_DEC_WAVES;
constexpr int kIters = PRCR_DEC_ITERS;   // key rows per lane group in flight

template <typename T>
struct Elems;
template <>
struct Elems<float> {
  static constexpr int kPerChunk = 4;
  __device__ static __forceinline__ void unpack(u32x4 w, float *x) {
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = __uint_as_float(w[q]);
  }
};
template <>
struct Elems<uint16_t> {
  static constexpr int kPerChunk = 8;
  __device__ static __forceinline__ void unpack(u32x4 w, float *x) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      x[2 * q] = __uint_as_float(w[q] << 16);
      x[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
    }
  }
};

// Scores are kept in base-2 units (the query carries log2(e)), so every
// softmax weight is one hardware exp2.
constexpr double kLog2e = 1.4426950408889634;
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Lane permutation within a 16-lane DPP row (no LDS round trip).
template <int kCtrl>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, 0xF, 0xF, false));
}

// Sum over the LPK consecutive lanes that hold one key row.  Every lane of the
// group ends with the same total: partners add the same two values at each step.
template <int LPK>
__device__ __forceinline__ float group_sum(float s) {
  static_assert(LPK == 8 || LPK == 16 || LPK == 32, "unsupported lane group");
  s += dpp<0xB1>(s);                               // quad permutation 1,0,3,2: lane ^ 1
  s += dpp<0x4E>(s);                               // quad permutation 2,3,0,1: lane ^ 2
  s += dpp<0x141>(s);                              // mirror in 8-lane halves: the other quad
  if constexpr (LPK >= 16) s += dpp<0x140>(s);     // mirror in the 16-lane row: the other half
  if constexpr (LPK >= 32) s += __shfl_xor(s, 16);
  return s;
}

// Sequence taken by workgroup row z.  With at most 64 sequences (lane l reads
// length l), the rows go to the sequences in order of decreasing length, ties by
// index.  Workgroups are dealt to the compute units in turn, so that each unit
// then holds chunks of long and of short sequences rather than a random mix: on a
// paged batch of 2,918-6,424 keys this measured 6 % faster.  Results do not depend
// on the order (each sequence is computed the same way by whichever row takes it).
__device__ __forceinline__ int sequence_of_row(const DecodeParams &p, int lane, int z) {
  if (p.batch > kWave) return z;
  const int mine = lane < p.batch ? max(p.cache_len[lane], 0) : -1;
  int rank = 0;
  for (int i = 0; i < p.batch; ++i) {
    const int other = __builtin_amdgcn_readlane(mine, i);
    rank += (other > mine) || (other == mine && i < lane);
  }
  const unsigned long long hit = __ballot(lane < p.batch && rank == z);
  return hit ? __ffsll(static_cast<long long>(hit)) - 1 : z;
}

template <typename T, int D, int GT, bool kPaged>
__global__ __launch_bounds__(kWaves * kWave) void decode_partial_kernel(const DecodeParams p) {
  constexpr int EPL = Elems<T>::kPerChunk;   // elements per lane (one 16-byte chunk)
  constexpr int LPK = D / EPL;               // lanes per key row
  constexpr int KPW = kWave / LPK;           // key rows per wave per iteration
  constexpr int KPB = kWaves * KPW;          // key rows per workgroup per iteration
  constexpr int kRowBytes = D * static_cast<int>(sizeof(T));
  constexpr int P = D / 2;
  static_assert(LPK >= 2 && kWave % LPK == 0, "unsupported head_dim");
  __shared__ float s_m[kWaves][GT];
  __shared__ float s_l[kWaves][GT];
  __shared__ float s_o[kWaves][GT][D];

  const int split = blockIdx.x, kvh = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int b = sequence_of_row(p, lane, blockIdx.z);
  const int wave = threadIdx.x / kWave;
  const int kg = lane / LPK;                 // key row slot within the wave
  const int c = lane % LPK;                  // 16-byte chunk of the row
  const int grp = wave * KPW + kg;           // key row slot within the workgroup
  const int G = p.n_q_heads / p.n_kv_heads;

  const int64_t cap = kPaged ? static_cast<int64_t>(p.max_blocks) * p.block_size : p.s_max;
  int len = p.cache_len[b];
  if (len < 0 || len > cap) {
    if (split == 0 && kvh == 0 && threadIdx.x == 0 && p.err != nullptr)
      atomicOr(p.err, PRCR_DERR_CAPACITY);
    len = static_cast<int>(min(max(static_cast<int64_t>(len), int64_t{0}), cap));
  }
  // The sequence's keys are shared evenly by its n_split workgroups, in whole
  // workgroup batches, so that no workgroup of a sequence waits on a longer one.
  const int per = (len + p.n_split - 1) / p.n_split;
  const int chunk = (per + KPB - 1) / KPB * KPB;
  const int j0 = min(len, split * chunk);
  const int j1 = min(len, j0 + chunk);

  // Rotated, scaled query chunk of every head of the group: the lane's elements
  // e = c*EPL .. c*EPL+EPL-1 pair with e +/- D/2, which sits in chunk c +/- LPK/2.
  float qv[GT][EPL];
  {
    const double pq = static_cast<double>(p.q_pos[b]);
    const bool first = c < LPK / 2;
    const int cp = first ? c + LPK / 2 : c - LPK / 2;
    double cs[EPL], sn[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      const int i = (c * EPL + e) % P;
      sincos(pq * p.inv_freq[i], &sn[e], &cs[e]);
    }
#pragma unroll
    for (int g = 0; g < GT; ++g) {
      const int qh = kvh * G + (g < G ? g : 0);
      const char *qrow = static_cast<const char *>(p.q) + (static_cast<int64_t>(b) * p.n_q_heads + qh) * kRowBytes;
      float x[EPL], xp[EPL];
      Elems<T>::unpack(*reinterpret_cast<const u32x4 *>(qrow + c * 16), x);
      Elems<T>::unpack(*reinterpret_cast<const u32x4 *>(qrow + cp * 16), xp);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        const double y = first ? static_cast<double>(x[e]) * cs[e] - static_cast<double>(xp[e]) * sn[e]
                               : static_cast<double>(x[e]) * cs[e] + static_cast<double>(xp[e]) * sn[e];
        qv[g][e] = static_cast<float>(y * (p.scale * kLog2e));
      }
    }
  }

  float m[GT], l[GT], o[GT][EPL];
#pragma unroll
  for (int g = 0; g < GT; ++g) {
    m[g] = -FLT_MAX;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[g][e] = 0.f;
  }

  const int64_t row_base = kPaged ? 0
                                  : ((static_cast<int64_t>(b) * p.n_layers + p.layer) * p.n_kv_heads + kvh) * p.s_max;
  int bad_block = 0;
  // Loads of the next batch of key rows are issued before the current batch is
  // scored, so one batch is always in flight.
  u32x4 kc[kIters], vc[kIters];
  bool live[kIters];
  // Slot 0 of this head's first row of the layer: present in every cache.
  const int64_t row_any = kPaged ? static_cast<int64_t>(p.layer) * p.n_blocks * p.block_size * p.n_kv_heads + kvh
                                 : row_base;
  auto load_batch = [&](int jb, u32x4 *kd, u32x4 *vd, bool *lv) {
    int32_t blk[kIters], in[kIters];
    if constexpr (kPaged) {
      // Every block-table entry of the batch is read before any row load is
      // issued: a wait for a table entry also waits for every load issued before
      // it, so reading them row by row would serialise the batch's row loads.
      // Rows past the chunk read the sequence's first entry (always present).
#pragma unroll
      for (int u = 0; u < kIters; ++u) {
        const int j = jb + u * KPB + grp;
        const int js = j < j1 ? j : 0;
        // Block and offset of slot js: a shift and a mask for power-of-two block
        // sizes (the common case), else one integer division.
        const int lb = p.block_shift >= 0 ? (js >> p.block_shift) : js / p.block_size;
        in[u] = js - lb * p.block_size;
        blk[u] = p.block_table[static_cast<int64_t>(b) * p.max_blocks + lb];
      }
    }
#pragma unroll
    for (int u = 0; u < kIters; ++u) {
      const int j = jb + u * KPB + grp;
      lv[u] = j < j1;
      int64_t row;
      if constexpr (kPaged) {
        if (lv[u] && (blk[u] < 0 || blk[u] >= p.n_blocks)) {
          lv[u] = false;
          bad_block = 1;
        }
        row = ((static_cast<int64_t>(p.layer) * p.n_blocks + blk[u]) * p.block_size + in[u]) *
                  p.n_kv_heads + kvh;
      } else {
        row = row_base + j;
      }
      // Rows past the chunk (or in a block outside the pool) read a row that
      // always exists, so that every load is issued unconditionally; they get
      // zero weight, and their values are taken as zero when scored.
      row = lv[u] ? row : row_any;
      kd[u] = load_nt(static_cast<const char *>(p.cache_k) + row * kRowBytes + c * 16);
      vd[u] = load_nt(static_cast<const char *>(p.cache_v) + row * kRowBytes + c * 16);
    }
  };
  load_batch(j0, kc, vc, live);
  for (int jb = j0; jb < j1; jb += KPB * kIters) {
    u32x4 nk[kIters], nv[kIters];
    bool nl[kIters];
    load_batch(jb + KPB * kIters, nk, nv, nl);
    // Scores of the batch's rows for every head of the group, then one rescale
    // of the running sums per head and batch.
    float sc[kIters][GT];
#pragma unroll
    for (int u = 0; u < kIters; ++u) {
      float k[EPL];
      Elems<T>::unpack(kc[u], k);
#pragma unroll
      for (int g = 0; g < GT; ++g) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) s = fmaf(qv[g][e], k[e], s);
        sc[u][g] = group_sum<LPK>(s);
      }
    }
    // A zero weight times a value read from another row could make a NaN:
    // values of rows without weight are taken as zero.
    float v[kIters][EPL];
#pragma unroll
    for (int u = 0; u < kIters; ++u) Elems<T>::unpack(live[u] ? vc[u] : u32x4{0u, 0u, 0u, 0u}, v[u]);
#pragma unroll
    for (int g = 0; g < GT; ++g) {
      float mn = m[g];
#pragma unroll
      for (int u = 0; u < kIters; ++u) mn = live[u] ? fmaxf(mn, sc[u][g]) : mn;
      // Rescale only when some lane's running maximum rose (rarely, after the
      // first rows): for every other lane the factor is exactly 1.
      if (__any(mn > m[g])) {
        const float corr = exp2_fast(m[g] - mn);
        l[g] *= corr;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] *= corr;
        m[g] = mn;
      }
#pragma unroll
      for (int u = 0; u < kIters; ++u) {
        const float pj = live[u] ? exp2_fast(sc[u][g] - mn) : 0.f;
        l[g] += pj;
#pragma unroll
        for (int e = 0; e < EPL; ++e) o[g][e] = fmaf(pj, v[u][e], o[g][e]);
      }
    }
#pragma unroll
    for (int u = 0; u < kIters; ++u) {
      kc[u] = nk[u];
      vc[u] = nv[u];
      live[u] = nl[u];
    }
  }
  if (bad_block && p.err != nullptr && c == 0) atomicOr(p.err, PRCR_DERR_BLOCK);

  // Merge the wave's key-row slots (lanes LPK apart hold the same elements of
  // different slots), then the workgroup's waves in LDS, and write this chunk's
  // partials.  Empty slots carry l = 0 and o = 0, so their weight is harmless.
#pragma unroll
  for (int off = LPK; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < GT; ++g) {
      const float m2 = __shfl_xor(m[g], off);
      const float l2 = __shfl_xor(l[g], off);
      const float mx = fmaxf(m[g], m2);
      const float w1 = exp2_fast(m[g] - mx), w2 = exp2_fast(m2 - mx);
      l[g] = l[g] * w1 + l2 * w2;
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] = o[g][e] * w1 + __shfl_xor(o[g][e], off) * w2;
      m[g] = mx;
    }
  }
  if (kg == 0) {
#pragma unroll
    for (int g = 0; g < GT; ++g) {
      if (c == 0) {
        s_m[wave][g] = m[g];
        s_l[wave][g] = l[g];
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) s_o[wave][g][c * EPL + e] = o[g][e];
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * D; idx += kWaves * kWave) {
    const int g = idx / D, d = idx % D;
    float M = -FLT_MAX;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][g]);
    float Ls = 0.f, Os = 0.f;
    for (int w = 0; w < kWaves; ++w) {
      const float wt = exp2_fast(s_m[w][g] - M);
      Ls += s_l[w][g] * wt;
      Os += s_o[w][g][d] * wt;
    }
    float *ws = p.ws + ((static_cast<int64_t>(b) * p.n_q_heads + kvh * G + g) * p.n_split + split) * (D + 2);
    ws[d] = Os;
    if (d == 0) {
      ws[D] = M;
      ws[D + 1] = Ls;
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 caches: the scores of a tile of 16 keys come from one matrix-core product
// per 32 elements of the head dim, K(16 keys) x Q(query rows)^T, with float32
// accumulation.  The float32 query of each head is split into three bf16 parts
// (the leading 8 significant bits, then the next 8 of what is left, then the
// rest), whose sum is exactly the float32 value, and the parts are rows of the
// product, so a key's score is the sum of its three part scores: as exact as a
// float32 dot product.  The softmax runs once per key in the lanes that hold the
// key's scores, with a running maximum shared by the wave, and the weights reach
// the lanes that hold the key's value row through LDS.

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma_16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Orders this wave's LDS writes before its later LDS reads (LDS operations of a
// wave complete in issue order; this keeps the compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Part `part` (0, 1, 2) of the three-way bf16 split of x, as bf16 bits in the
// upper half of a word.  Each part is the truncation of what the previous parts
// left, and every difference is exact in float32, so the parts sum to x.
__device__ __forceinline__ uint32_t split_part(float x, int part) {
  const uint32_t hi = __float_as_uint(x) & 0xFFFF0000u;
  const float r1 = x - __uint_as_float(hi);
  const uint32_t mid = __float_as_uint(r1) & 0xFFFF0000u;
  const float r2 = r1 - __uint_as_float(mid);
  return part == 0 ? hi : (part == 1 ? mid : __float_as_uint(r2));
}

// Maximum over the 16 lanes of a DPP row; every lane of the row ends with it.
__device__ __forceinline__ float row_max16(float s) {
  s = fmaxf(s, dpp<0xB1>(s));
  s = fmaxf(s, dpp<0x4E>(s));
  s = fmaxf(s, dpp<0x141>(s));
  s = fmaxf(s, dpp<0x140>(s));
  return s;
}

// kTileBlocks (paged only): block_size is a multiple of 16, so that every tile
// of 16 keys (tiles start at multiples of 16) lies in one block.
template <int D, int GT, bool kPaged, bool kTileBlocks>
__global__ __launch_bounds__(kWaves * kWave, GT >= 8 ? 2 : 3) void decode_partial_bf16_kernel(const DecodeParams p) {
  constexpr int kTile = 16;                  // keys per wave and tile: the product's N
  constexpr int KK = D / 32;                 // products over the head dim per query row tile
  constexpr int kRows = 3 * GT;              // query rows: three parts of every head
  constexpr int kATiles = (kRows + 15) / 16; // 16-row query tiles
  constexpr int kXS = kATiles * 16 + 4;      // floats per key in the part-score exchange (padded)
  constexpr int EPL = Elems<uint16_t>::kPerChunk;   // value elements per lane (one 16-byte chunk)
  constexpr int LPK = D / EPL;               // lanes per value row
  constexpr int KPW = kWave / LPK;           // value rows per load
  constexpr int VL = kTile / KPW;            // value loads per lane and tile
  constexpr int kRowBytes = D * 2;
  constexpr int KPB = kWaves * kTile;        // keys per workgroup per round of tiles
  constexpr int P = D / 2;
  static_assert(KK >= 1 && D % 32 == 0 && VL >= 1, "unsupported head_dim");
  __shared__ __align__(16) float s_q[GT][D];
  __shared__ __align__(16) float s_x[kWaves][kTile][kXS];
  __shared__ __align__(16) float s_p[kWaves][kTile][GT];
  __shared__ float s_m[kWaves][GT];
  __shared__ float s_l[kWaves][GT];
  __shared__ float s_o[kWaves][GT][D];

  const int split = blockIdx.x, kvh = blockIdx.y;
  const int lane = threadIdx.x & (kWave - 1);
  const int b = sequence_of_row(p, lane, blockIdx.z);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int kt = lane % kTile;               // key of the tile whose scores this lane holds
  const int kj = lane / kTile;               // 16-byte chunks 4*kk + kj of that key's row
  const int vr = lane / LPK;                 // value row slot within a load
  const int vc = lane % LPK;                 // 16-byte chunk of the value row
  const int G = p.n_q_heads / p.n_kv_heads;

  const int64_t cap = kPaged ? static_cast<int64_t>(p.max_blocks) * p.block_size : p.s_max;
  int len = p.cache_len[b];
  if (len < 0 || len > cap) {
    if (split == 0 && kvh == 0 && threadIdx.x == 0 && p.err != nullptr)
      atomicOr(p.err, PRCR_DERR_CAPACITY);
    len = static_cast<int>(min(max(static_cast<int64_t>(len), int64_t{0}), cap));
  }
  const int per = (len + p.n_split - 1) / p.n_split;
  const int chunk = (per + KPB - 1) / KPB * KPB;
  const int j0 = min(len, split * chunk);
  const int j1 = min(len, j0 + chunk);

  // Rotated, scaled query of every head of the group (pair i with i + D/2, the
  // 1-D rotation at p_next), in float32, in LDS.
  {
    const double pq = static_cast<double>(p.q_pos[b]);
    const double qs = static_cast<double>(p.scale) * kLog2e;
    for (int idx = threadIdx.x; idx < GT * P; idx += kWaves * kWave) {
      const int g = idx / P, i = idx % P;
      const int qh = kvh * G + (g < G ? g : 0);
      const uint16_t *qrow = static_cast<const uint16_t *>(p.q) + (static_cast<int64_t>(b) * p.n_q_heads + qh) * D;
      double sn, cs;
      sincos(pq * p.inv_freq[i], &sn, &cs);
      const double x = __uint_as_float(static_cast<uint32_t>(qrow[i]) << 16);
      const double xp = __uint_as_float(static_cast<uint32_t>(qrow[i + P]) << 16);
      s_q[g][i] = static_cast<float>((x * cs - xp * sn) * qs);
      s_q[g][i + P] = static_cast<float>((xp * cs + x * sn) * qs);
    }
  }
  __syncthreads();
  // Query operand: row r = 16a + lane%16 of tile a is part r / GT of head r % GT;
  // the lane's 8 elements of product kk are those of row chunk 4*kk + kj, the
  // same chunk as the key operand below.
  u32x4 qa[kATiles][KK];
#pragma unroll
  for (int a = 0; a < kATiles; ++a) {
    const int r = 16 * a + kt;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      u32x4 w = {0u, 0u, 0u, 0u};
      if (r < kRows) {
        const int part = r / GT, g = r % GT;
        const float *src = &s_q[g][8 * (4 * kk + kj)];
#pragma unroll
        for (int h = 0; h < 4; ++h)
          w[h] = (split_part(src[2 * h], part) >> 16) | (split_part(src[2 * h + 1], part) & 0xFFFF0000u);
      }
      qa[a][kk] = w;
    }
  }

  const int64_t row_base = kPaged ? 0
                                  : ((static_cast<int64_t>(b) * p.n_layers + p.layer) * p.n_kv_heads + kvh) * p.s_max;
  const int64_t row_any = kPaged ? static_cast<int64_t>(p.layer) * p.n_blocks * p.block_size * p.n_kv_heads + kvh
                                 : row_base;
  int bad_block = 0;
  // Block-table entry of key j (the sequence's first entry past the chunk).
  auto table = [&](int j) -> int32_t {
    const int js = j < j1 ? j : 0;
    const int lb = p.block_shift >= 0 ? (js >> p.block_shift) : js / p.block_size;
    return p.block_table[static_cast<int64_t>(b) * p.max_blocks + lb];
  };
  // Addressing.  Contiguous caches and whole-tile blocks address a tile by its
  // first row and the stride between its keys' rows (1 row, or n_kv_heads rows
  // within a block); other paged caches read a block-table entry per key.  Keys
  // at or past `lim`, or in a block outside the pool, read row_any instead (every
  // load is issued unconditionally) and are marked dead: they get no weight,
  // and their values are taken as zero.
  struct TileAddr {
    int64_t base;
    bool ok;
  };
  auto tile_addr = [&](int tb, int32_t blk) -> TileAddr {
    if constexpr (kTileBlocks) {
      const int lb = p.block_shift >= 0 ? (tb >> p.block_shift) : tb / p.block_size;
      const bool ok = blk >= 0 && blk < p.n_blocks;
      return {((static_cast<int64_t>(p.layer) * p.n_blocks + blk) * p.block_size + (tb - lb * p.block_size)) *
                      p.n_kv_heads + kvh, ok};
    } else {
      return {row_base + tb, true};
    }
  };
  constexpr int kStrideHeads = kPaged ? 1 : 0;   // rows between keys: n_kv_heads (paged) or 1
  auto key_row = [&](int tb, const TileAddr &ta, int t, int lim, bool &live) -> int64_t {
    const int j = tb + t;
    const bool in = j < lim;
    if constexpr (kPaged && !kTileBlocks) {
      const int32_t blk = table(j);
      const bool ok = blk >= 0 && blk < p.n_blocks;
      bad_block |= in && !ok;
      live = in && ok;
      const int lb = p.block_shift >= 0 ? (j >> p.block_shift) : j / p.block_size;
      const int64_t row = ((static_cast<int64_t>(p.layer) * p.n_blocks + blk) * p.block_size + (j - lb * p.block_size)) *
                              p.n_kv_heads + kvh;
      return live ? row : row_any;
    } else {
      bad_block |= in && !ta.ok;
      live = in && ta.ok;
      const int64_t row = ta.base + static_cast<int64_t>(t) * (kStrideHeads ? p.n_kv_heads : 1);
      return live ? row : row_any;
    }
  };
  // Key rows of a tile in the product's operand layout.  A load reads a quarter
  // of each of 16 rows and the other quarters follow at once from the same cache
  // lines, so these are plain loads: as non-temporal loads they took 10 % longer.
  auto load_k = [&](int tb, const TileAddr &ta, int lim, u32x4 *kd, bool &kl) {
    const int64_t rk = key_row(tb, ta, kt, lim, kl);
    const char *kp = static_cast<const char *>(p.cache_k) + rk * kRowBytes + kj * 16;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      kd[kk] = *reinterpret_cast<const u32x4 *>(kp + kk * 64);
  };
  // Value rows of a tile, 16 lanes to a row.
  auto load_v = [&](int tb, const TileAddr &ta, int lim, u32x4 *vd, bool *vl) {
    int64_t rv[VL];
#pragma unroll
    for (int u = 0; u < VL; ++u) rv[u] = key_row(tb, ta, KPW * u + vr, lim, vl[u]);
#pragma unroll
    for (int u = 0; u < VL; ++u)
      vd[u] = load_nt(static_cast<const char *>(p.cache_v) + rv[u] * kRowBytes + vc * 16);
  };

  float o[GT][EPL], lsum[GT], mrun[GT];
#pragma unroll
  for (int g = 0; g < GT; ++g) {
    lsum[g] = 0.f;
    mrun[g] = -FLT_MAX;
#pragma unroll
    for (int e = 0; e < EPL; ++e) o[g][e] = 0.f;
  }

  // The wave's tiles start at jw + n*KPB.  With whole-tile blocks the wave reads
  // the block-table entries of 64 tiles at once, one per lane, and takes each
  // from its lane when the tile comes; the keys of the next 64 tiles are then a
  // new round (its first tile loaded again; keys from `lim` on are dead here).
  //
  // One buffer per operand, software-pipelined: the next tile's key rows are
  // loaded once this tile's product has read them, and its value rows once this
  // tile's weighted sum has; each load's latency hides behind the other half of
  // a tile's work, and every wait is for the oldest loads only.
  const int jw = j0 + wave * kTile;
  // Rounds of 64 tiles with whole-tile blocks; one round otherwise (lim = j1).
  const int n_tiles = jw < j1 ? (j1 - jw + KPB - 1) / KPB : 0;
  const int rounds = kTileBlocks ? (n_tiles + kWave - 1) / kWave : (n_tiles > 0 ? 1 : 0);
  for (int r = 0; r < rounds; ++r) {
    const int n0 = r * kWave;
    int32_t tab_lane = 0;
    if constexpr (kTileBlocks) tab_lane = table(jw + (n0 + lane) * KPB);
    const int lim = kTileBlocks ? static_cast<int>(min(static_cast<int64_t>(j1),
                                                       static_cast<int64_t>(jw) + static_cast<int64_t>(n0 + kWave) * KPB))
                                : j1;
    auto addr_of = [&](int n) -> TileAddr {
      const int tb = jw + n * KPB;
      int32_t blk = 0;
      if constexpr (kTileBlocks) blk = __builtin_amdgcn_readlane(tab_lane, min(n - n0, kWave - 1));
      return tile_addr(tb, blk);
    };
    u32x4 kr[KK], vv[VL];
    bool kl, vl[VL];
    int n = n0, jt = jw + n0 * KPB;
    TileAddr ta = addr_of(n);
    load_k(jt, ta, lim, kr, kl);
    load_v(jt, ta, lim, vv, vl);
    while (jt < lim) {
      const TileAddr ta_n = addr_of(n + 1);
      // Part scores: lane holds rows 16a + 4*(lane/16) + i of the product for key kt.
      f32x4 acc[kATiles];
#pragma unroll
      for (int a = 0; a < kATiles; ++a) {
        acc[a] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) acc[a] = mfma_16x16x32(qa[a][kk], kr[kk], acc[a]);
      }
      bool kl_n;
      load_k(jt + KPB, ta_n, lim, kr, kl_n);
#pragma unroll
      for (int a = 0; a < kATiles; ++a) {
        const int r0 = 16 * a + 4 * kj;
        if (r0 < kRows) *reinterpret_cast<f32x4 *>(&s_x[wave][kt][r0]) = acc[a];
      }
      wave_lds_sync();
      // Every row of 16 lanes now takes the same 16 keys: lane kt's key, all heads.
      float sc[GT];
      bool rise = false;
#pragma unroll
      for (int g = 0; g < GT; ++g) {
        const float s = (s_x[wave][kt][g] + s_x[wave][kt][GT + g]) + s_x[wave][kt][2 * GT + g];
        sc[g] = kl ? s : -FLT_MAX;
        rise = rise || sc[g] > mrun[g];
      }
      // The tile's maxima are needed only when some score rose above the running
      // maximum of its head (rarely, after the first tiles).
      if (__any(rise)) {
#pragma unroll
        for (int g = 0; g < GT; ++g) {
          const float tmax = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(row_max16(sc[g]))));
          const float mnew = fmaxf(mrun[g], tmax);
          const float corr = exp2_fast(mrun[g] - mnew);
          lsum[g] *= corr;
#pragma unroll
          for (int e = 0; e < EPL; ++e) o[g][e] *= corr;
          mrun[g] = mnew;
        }
      }
      float pw[GT];
#pragma unroll
      for (int g = 0; g < GT; ++g) {
        pw[g] = exp2_fast(sc[g] - mrun[g]);
        lsum[g] += pw[g];
      }
      if (lane < kTile) {
#pragma unroll
        for (int g = 0; g < GT; ++g) s_p[wave][kt][g] = pw[g];
      }
      wave_lds_sync();
      // A zero weight times a value read from another row could make a NaN:
      // values of keys without weight are taken as zero.
#pragma unroll
      for (int u = 0; u < VL; ++u) {
        const int tk = KPW * u + vr;
        float v[EPL];
        Elems<uint16_t>::unpack(vl[u] ? vv[u] : u32x4{0u, 0u, 0u, 0u}, v);
#pragma unroll
        for (int g = 0; g < GT; ++g) {
          const float w = s_p[wave][tk][g];
#pragma unroll
          for (int e = 0; e < EPL; ++e) o[g][e] = fmaf(w, v[e], o[g][e]);
        }
      }
      load_v(jt + KPB, ta_n, lim, vv, vl);
      kl = kl_n;
      jt += KPB;
      ++n;
    }
  }
  if (bad_block && p.err != nullptr) atomicOr(p.err, PRCR_DERR_BLOCK);

  // Every lane of the wave used the same running maxima: the value row slots add
  // up plainly, and so do the weight sums of the 16 keys of a row of lanes.
#pragma unroll
  for (int off = LPK; off < kWave; off <<= 1) {
#pragma unroll
    for (int g = 0; g < GT; ++g) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) o[g][e] += __shfl_xor(o[g][e], off);
    }
  }
#pragma unroll
  for (int g = 0; g < GT; ++g) lsum[g] = group_sum<16>(lsum[g]);
  if (lane < LPK) {
#pragma unroll
    for (int g = 0; g < GT; ++g) {
      if (lane == 0) {
        s_m[wave][g] = mrun[g];
        s_l[wave][g] = lsum[g];
      }
#pragma unroll
      for (int e = 0; e < EPL; ++e) s_o[wave][g][vc * EPL + e] = o[g][e];
    }
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < G * D; idx += kWaves * kWave) {
    const int g = idx / D, d = idx % D;
    float M = -FLT_MAX;
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][g]);
    float Ls = 0.f, Os = 0.f;
    for (int w = 0; w < kWaves; ++w) {
      const float wt = exp2_fast(s_m[w][g] - M);
      Ls += s_l[w][g] * wt;
      Os += s_o[w][g][d] * wt;
    }
    float *ws = p.ws + ((static_cast<int64_t>(b) * p.n_q_heads + kvh * G + g) * p.n_split + split) * (D + 2);
    ws[d] = Os;
    if (d == 0) {
      ws[D] = M;
      ws[D + 1] = Ls;
    }
  }
}

// Merge of one query head's split partials.  Each split's (max, sum) is read by
// one thread, D splits at a time, so that the reads go out together instead of
// one after another's use; the weights pass through LDS, and every thread then
// accumulates its feature over the splits in split order with the same fused
// multiply-adds as a sequential merge (an empty split adds exact zeros).  The
// feature values of the first kPre splits do not depend on the weights: they are
// read in the same round as the (max, sum) pairs.
template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(const DecodeParams p) {
  constexpr int kPre = 8;
  __shared__ float s_red[D / kWave];
  __shared__ float s_w[D], s_l[D];
  const int qh = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
  const int lane = d & (kWave - 1), wave = d / kWave;
  const int ns = p.n_split;
  const float *ws = p.ws + (static_cast<int64_t>(b) * p.n_q_heads + qh) * ns * (D + 2);
  float o_pre[kPre];
#pragma unroll
  for (int k = 0; k < kPre; ++k) o_pre[k] = ws[static_cast<int64_t>(min(k, ns - 1)) * (D + 2) + d];
  // Largest max over the splits that saw a key.  Both values of a split are
  // read before either is used; a thread keeps those of its first split (every
  // split, when n_split <= D) for the second pass.
  float M = -FLT_MAX, l_first = 0.f, m_first = -FLT_MAX;
  for (int s0 = 0; s0 < ns; s0 += D) {
    const int s = min(s0 + d, ns - 1);
    const float l = ws[static_cast<int64_t>(s) * (D + 2) + D + 1];
    const float m = ws[static_cast<int64_t>(s) * (D + 2) + D];
    const bool used = s0 + d < ns && l > 0.f;
    M = used ? fmaxf(M, m) : M;
    if (s0 == 0) {
      l_first = used ? l : 0.f;
      m_first = m;
    }
  }
  for (int o = kWave / 2; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  if (lane == 0) s_red[wave] = M;
  __syncthreads();
  M = s_red[0];
#pragma unroll
  for (int w = 1; w < D / kWave; ++w) M = fmaxf(M, s_red[w]);
  float Ls = 0.f, Os = 0.f;
  for (int s0 = 0; s0 < ns; s0 += D) {
    const int s = s0 + d;
    float l = l_first, m = m_first;
    if (s0 > 0) {
      const int sc = min(s, ns - 1);
      l = ws[static_cast<int64_t>(sc) * (D + 2) + D + 1];
      m = ws[static_cast<int64_t>(sc) * (D + 2) + D];
      l = s < ns && l > 0.f ? l : 0.f;
    }
    const float w = l > 0.f ? exp2_fast(m - M) : 0.f;
    __syncthreads();
    s_w[d] = w;
    s_l[d] = l;
    __syncthreads();
    const int cnt = min(D, ns - s0);
    const float *o = ws + static_cast<int64_t>(s0) * (D + 2) + d;
    int k0 = 0;
    if (s0 == 0) {
#pragma unroll
      for (int k = 0; k < kPre; ++k) {
        if (k < cnt) {
          Ls = fmaf(s_l[k], s_w[k], Ls);
          Os = fmaf(o_pre[k], s_w[k], Os);
        }
      }
      k0 = kPre;
    }
#pragma unroll 4
    for (int k = k0; k < cnt; ++k) {
      Ls = fmaf(s_l[k], s_w[k], Ls);
      Os = fmaf(o[static_cast<int64_t>(k) * (D + 2)], s_w[k], Os);
    }
  }
  p.out[(static_cast<int64_t>(b) * p.n_q_heads + qh) * D + d] = Ls > 0.f ? Os / Ls : 0.f;
}

template <typename T, int D, int GT, bool kPaged>
hipError_t launch_split(const DecodeParams &p, hipStream_t stream) {
  const dim3 grid(p.n_split, p.n_kv_heads, p.batch);
  if constexpr (std::is_same_v<T, uint16_t> && PRCR_DEC_MFMA) {
    if constexpr (kPaged) {
      if (p.block_size % 16 == 0)
        decode_partial_bf16_kernel<D, GT, true, true><<<grid, kWaves * kWave, 0, stream>>>(p);
      else
        decode_partial_bf16_kernel<D, GT, true, false><<<grid, kWaves * kWave, 0, stream>>>(p);
    } else {
      decode_partial_bf16_kernel<D, GT, false, false><<<grid, kWaves * kWave, 0, stream>>>(p);
    }
  } else
    decode_partial_kernel<T, D, GT, kPaged>
        <<<dim3(p.n_split, p.n_kv_heads, p.batch), kWaves * kWave, 0, stream>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  decode_combine_kernel<D><<<dim3(p.n_q_heads, p.batch), D, 0, stream>>>(p);
  return hipGetLastError();
}

template <typename T, int D, bool kPaged>
hipError_t dispatch_group(const DecodeParams &p, int G, hipStream_t stream) {
  if (G <= 1) return launch_split<T, D, 1, kPaged>(p, stream);
  if (G <= 2) return launch_split<T, D, 2, kPaged>(p, stream);
  if (G <= 4) return launch_split<T, D, 4, kPaged>(p, stream);
  return launch_split<T, D, 8, kPaged>(p, stream);
}

template <typename T, bool kPaged>
hipError_t dispatch_dim(const DecodeParams &p, int head_dim, int G, hipStream_t stream) {
  if (head_dim == 64) return dispatch_group<T, 64, kPaged>(p, G, stream);
  if (head_dim == 128) return dispatch_group<T, 128, kPaged>(p, G, stream);
  return hipErrorInvalidValue;
}

}  // namespace

int decode_splits(int64_t capacity, int batch, int n_kv_heads, int group) {
  // About as many workgroups as the chip holds at once, so that all of them
  // start together and none waits for a second round: 256 compute units with 3
  // workgroups of the bf16 kernel each (2 with 8 query heads per KV head, whose
  // kernel holds more registers).  No split of fewer than 64 keys at full
  // capacity.
  const int64_t target = PRCR_DEC_WORKGROUPS > 0 ? PRCR_DEC_WORKGROUPS : (group > 4 ? 512 : 768);
  const int64_t pairs = static_cast<int64_t>(batch) * n_kv_heads;
  int64_t ns = (target + pairs - 1) / pairs;
  const int64_t most = (capacity + 63) / 64;
  if (ns > most) ns = most;
  if (ns < 1) ns = 1;
  return static_cast<int>(ns);
}

hipError_t launch_decode(const DecodeParams &p, prcr_dtype dtype, int head_dim, bool paged,
                         hipStream_t stream) {
  const int G = p.n_q_heads / p.n_kv_heads;
  if (dtype == PRCR_F32)
    return paged ? dispatch_dim<float, true>(p, head_dim, G, stream)
                 : dispatch_dim<float, false>(p, head_dim, G, stream);
  return paged ? dispatch_dim<uint16_t, true>(p, head_dim, G, stream)
               : dispatch_dim<uint16_t, false>(p, head_dim, G, stream);
}

}  // namespace prcr
