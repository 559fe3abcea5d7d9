// Prefill capture fused with rotary (the step before a revisit): for one layer,
// read each prompt token's pre-rotary K/V rows once and
//   * write the rotated key and the value into the standard decoder cache at the
//     token's original position ids, Eq. (4), and
//   * for visual tokens, write the raw rows into the Raw Visual Evidence Memory,
//     Eq. (6)-(7) (optionally with the token's coordinates).
//
// One wavefront covers PRCR_PF_ITERS x (rows per iteration) consecutive
// (sequence, token, head) rows of the layer (8 at bf16, d 128: one token's 8
// heads); a lane owns one 16-byte chunk of each half of a row, as in the rebind
// kernel.  A wave moves one batch of rows, so its latency is mostly the chain of
// dependent loads before its stores: the kernel keeps that chain at two rounds
// (three for a paged destination).
#include <climits>
#include <cmath>

#include "prcr_internal.h"
#include "rotary.h"

namespace prcr {
namespace {

#ifndef PRCR_PF_ITERS
#define PRCR_PF_ITERS 1
#endif
constexpr int kWaves = 4;
constexpr int kIters = PRCR_PF_ITERS;

// kTPI: whole tokens per iteration of RPI rows.  1: n_kv_heads is a multiple of
// the rows per iteration, so an iteration's rows are heads of one token;
// validity and slot are then uniform across the wave, and one sincos per lane
// shared by shuffles covers the token.  2: the rows per iteration are two
// tokens' heads (n_kv_heads = RPI / 2); the wave evaluates each token's P angles
// once (one or two per lane, while every lane is active) and shares them by shuffles.
// 0: each lane evaluates the E pairs of its own row.
template <typename T, int D, class Map, bool kPaged, int kTPI>
__global__ __launch_bounds__(kWaves * kWave) void prefill_capture_kernel(const PrefillParams p) {
  constexpr int P = D / 2;
  constexpr int E = Store<T>::kPerChunk;
  constexpr int LPR = P / E;
  constexpr int RPI = kWave / LPR;
  constexpr int kRowBytes = D * static_cast<int>(sizeof(T));
  constexpr int kHalfBytes = kRowBytes / 2;
  static_assert(Map::kPairs == P, "axis map does not match head_dim");

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = threadIdx.x / kWave;
  const int H = p.n_kv_heads;
  const int64_t rows_all = static_cast<int64_t>(p.batch) * p.s_src * H;
  const int64_t base = (static_cast<int64_t>(blockIdx.x) * kWaves + wave) * (RPI * kIters);
  if (base >= rows_all) return;
  const int r = lane / LPR;
  const int c = lane % LPR;

  // The wave's loads are issued in two rounds, from indices that are always in
  // range: first each row's sequence length, then together the raw rows of the
  // live rows (those below n_tokens) and, per row, its token's position ids,
  // visual index and sequence values, plus this lane's rotary frequency.  Vector
  // loads complete in issue order, so a load issued only after another's value
  // is used waits a round trip more.  Only a paged destination's block-table
  // entry waits on these.
  int rb[kIters], rs[kIters], rh[kIters];
  int32_t nt[kIters];
  int64_t Rc[kIters];
  bool inr[kIters];
#pragma unroll
  for (int u = 0; u < kIters; ++u) {
    const int64_t R = base + u * RPI + r;
    inr[u] = R < rows_all;
    Rc[u] = inr[u] ? R : rows_all - 1;
    rb[u] = static_cast<int>(Rc[u] / (static_cast<int64_t>(p.s_src) * H));
    const int64_t rem = Rc[u] - static_cast<int64_t>(rb[u]) * p.s_src * H;
    rs[u] = static_cast<int>(rem / H);
    rh[u] = static_cast<int>(rem - static_cast<int64_t>(rs[u]) * H);
    nt[u] = p.n_tokens[rb[u]];
  }
  const double inv_lane = p.inv_freq[lane % P];
  u32x4 kl[kIters], kh[kIters], vl[kIters], vh[kIters];
  int32_t cst[kIters], vis[kIters], nvis[kIters], pid[kIters][3];
  bool live[kIters];
#pragma unroll
  for (int u = 0; u < kIters; ++u) {
    const int64_t tok = static_cast<int64_t>(rb[u]) * p.s_src + rs[u];
    cst[u] = p.cache_start[rb[u]];
    nvis[u] = p.n_visual[rb[u]];
    vis[u] = p.vis_index[tok];
    pid[u][0] = p.pos[3 * tok + 0];
    pid[u][1] = p.pos[3 * tok + 1];
    pid[u][2] = p.pos[3 * tok + 2];
    live[u] = inr[u] && rs[u] < min(max(nt[u], 0), p.s_src);
    if (live[u]) {
      const size_t o = static_cast<size_t>(Rc[u]) * kRowBytes + c * 16;
      kl[u] = load_nt(static_cast<const char *>(p.raw_k) + o);
      kh[u] = load_nt(static_cast<const char *>(p.raw_k) + o + kHalfBytes);
      vl[u] = load_nt(static_cast<const char *>(p.raw_v) + o);
      vh[u] = load_nt(static_cast<const char *>(p.raw_v) + o + kHalfBytes);
    }
  }
  // Per-row rotation: the lane's E frequencies, taken from the lanes that hold
  // them while every lane is still active.
  double inv[kTPI == 0 ? E : 1];
  if constexpr (kTPI == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) inv[e] = __shfl(inv_lane, c * E + e);
  }

#pragma unroll
  for (int u = 0; u < kIters; ++u) {
    const int b = rb[u], s = rs[u], h = rh[u];
    // Two tokens per iteration: lane l evaluates pair l % P of token (64 j + l) / P
    // for j < NS (position ids from the first lane of the token's first row), then
    // each lane gathers its own row's E pairs.
    double cs_it[kTPI >= 2 ? E : 1], sn_it[kTPI >= 2 ? E : 1];
    if constexpr (kTPI >= 2) {
      constexpr int NS = (kTPI * P + kWave - 1) / kWave;
      constexpr int kLanesPerTok = kWave / kTPI;
      const int ax = Map::axis(lane % P);
      double cv[NS], sv[NS];
#pragma unroll
      for (int j = 0; j < NS; ++j) {
        const int tk = min((j * kWave + lane) / P, kTPI - 1);
        const int src = tk * kLanesPerTok;
        const int p0 = __shfl(pid[u][0], src), p1 = __shfl(pid[u][1], src), p2 = __shfl(pid[u][2], src);
        const double pa = ax == 0 ? p0 : (ax == 1 ? p1 : p2);
        sincos(pa * inv_lane, &sv[j], &cv[j]);
      }
      const int tk_me = lane / kLanesPerTok;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int g = tk_me * P + c * E + e;
        const int src = g % kWave, slot = g / kWave;
#pragma unroll
        for (int j = 0; j < NS; ++j) {
          const double cj = __shfl(cv[j], src), sj = __shfl(sv[j], src);
          if (slot == j) {
            cs_it[e] = cj;
            sn_it[e] = sj;
          }
        }
      }
    }
    if (inr[u] && (nt[u] < 0 || nt[u] > p.s_src) && s == 0 && h == 0 && c == 0 && p.err)
      atomicOr(p.err, PRCR_DERR_INDEX);
    if (!live[u]) continue;
    const double pt = pid[u][0], ph = pid[u][1], pw = pid[u][2];

    // Standard cache: rotated key and value at slot cache_start[b] + s (Eq. (4)).
    const int64_t slot = static_cast<int64_t>(cst[u]) + s;
    int64_t d = -1;
    int flag = 0;
    if constexpr (kPaged) {
      const int64_t lb = slot >= 0 ? slot / p.block_size : -1;
      if (lb < 0 || lb >= p.max_blocks) {
        flag = PRCR_DERR_CAPACITY;
      } else {
        const int64_t blk = p.block_table[static_cast<int64_t>(b) * p.max_blocks + lb];
        if (blk < 0 || blk >= p.n_blocks) {
          flag = PRCR_DERR_BLOCK;
        } else {
          const int64_t off = slot - lb * p.block_size;
          d = ((static_cast<int64_t>(p.layer) * p.n_blocks + blk) * p.block_size + off) * H + h;
        }
      }
    } else {
      if (slot < 0 || slot >= p.s_max)
        flag = PRCR_DERR_CAPACITY;
      else
        d = ((static_cast<int64_t>(b) * p.n_layers + p.layer) * H + h) * p.s_max + slot;
    }
    if (d >= 0) {
      double cs[E], sn[E];
      if constexpr (kTPI >= 2) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          cs[e] = cs_it[e];
          sn[e] = sn_it[e];
        }
      } else if constexpr (kTPI == 1) {
        // All rows of this iteration belong to one token: lane i evaluates pair i
        // (mod P) and each lane gathers its E pairs with shuffles.
        const int pair = lane % P;
        const int ax = Map::axis(pair);
        double sv, cv;
        sincos((ax == 0 ? pt : (ax == 1 ? ph : pw)) * inv_lane, &sv, &cv);
#pragma unroll
        for (int e = 0; e < E; ++e) {
          cs[e] = __shfl(cv, c * E + e);
          sn[e] = __shfl(sv, c * E + e);
        }
      } else {
#pragma unroll
        for (int e = 0; e < E; ++e) {
          const int ax = Map::axis(c * E + e);
          sincos((ax == 0 ? pt : (ax == 1 ? ph : pw)) * inv[e], &sn[e], &cs[e]);
        }
      }
      u32x4 ol, oh;
      Store<T>::rotate(kl[u], kh[u], cs, sn, ol, oh);
      char *ck = static_cast<char *>(p.cache_k) + d * kRowBytes + c * 16;
      char *cv = static_cast<char *>(p.cache_v) + d * kRowBytes + c * 16;
      store_nt(ck, ol);
      store_nt(ck + kHalfBytes, oh);
      store_nt(cv, vl[u]);
      store_nt(cv + kHalfBytes, vh[u]);
    }

    // Raw Visual Evidence Memory: raw rows of visual tokens (Eq. (6)-(7)).
    const int m = vis[u];
    if (m >= 0) {
      if (m >= p.max_visual || m >= nvis[u]) {
        flag |= PRCR_DERR_INDEX;
      } else {
        const size_t mo = (((static_cast<size_t>(b) * p.max_visual + m) * p.n_layers + p.layer) * H + h) *
                              kRowBytes + c * 16;
        char *mk = static_cast<char *>(p.mem_k) + mo;
        store_nt(mk, kl[u]);
        store_nt(mk + kHalfBytes, kh[u]);
        if (p.mem_v != nullptr) {
          char *mv = static_cast<char *>(p.mem_v) + mo;
          store_nt(mv, vl[u]);
          store_nt(mv + kHalfBytes, vh[u]);
        } else if (p.v_slot != nullptr && h == 0 && c == 0) {
          // key-only memory: the value rows stay in this cache slot (-1 if the
          // slot could not be written)
          p.v_slot[static_cast<int64_t>(b) * p.max_visual + m] = d >= 0 ? static_cast<int32_t>(slot) : -1;
        }
        if (p.write_coords && h == 0 && c == 0) {
          int32_t *co = p.coords + (static_cast<int64_t>(b) * p.max_visual + m) * 3;
          co[0] = pid[u][0];
          co[1] = pid[u][1];
          co[2] = pid[u][2];
        }
      }
    }
    if (flag != 0 && c == 0 && p.err != nullptr) atomicOr(p.err, flag);
  }
}

template <typename T, int D, class Map, bool kPaged>
hipError_t launch_one(const PrefillParams &p, hipStream_t stream) {
  constexpr int LPR = (D / 2) / Store<T>::kPerChunk;
  constexpr int RPI = kWave / LPR;
  const int64_t rows_all = static_cast<int64_t>(p.batch) * p.s_src * p.n_kv_heads;
  const int64_t per_block = static_cast<int64_t>(kWaves) * RPI * kIters;
  int64_t blocks = (rows_all + per_block - 1) / per_block;
  if (blocks < 1) blocks = 1;
  if (!grid_fits(blocks, kWaves * kWave)) return hipErrorInvalidConfiguration;
  constexpr int P = D / 2;
  const dim3 grid(static_cast<unsigned>(blocks)), block(kWaves * kWave);
  const int H = p.n_kv_heads;
  const int tpi = RPI % H == 0 ? RPI / H : 0;
  if (H % RPI == 0)
    prefill_capture_kernel<T, D, Map, kPaged, 1><<<grid, block, 0, stream>>>(p);
  else if (tpi == 2 && 2 * P <= 2 * kWave)
    prefill_capture_kernel<T, D, Map, kPaged, 2><<<grid, block, 0, stream>>>(p);
  else
    prefill_capture_kernel<T, D, Map, kPaged, 0><<<grid, block, 0, stream>>>(p);
  return hipGetLastError();
}

template <typename T, bool kPaged>
hipError_t dispatch_map(const PrefillParams &p, int head_dim, AxisMapId map, hipStream_t stream) {
  if (head_dim == 64) {
    if (map == AxisMapId::kS_8_12_12) return launch_one<T, 64, Sectioned<8, 12, 12>, kPaged>(p, stream);
    if (map == AxisMapId::kI_11_11_10) return launch_one<T, 64, Interleaved<11, 11, 10>, kPaged>(p, stream);
    if (map == AxisMapId::kS_32_0_0) return launch_one<T, 64, Sectioned<32, 0, 0>, kPaged>(p, stream);
  } else if (head_dim == 128) {
    if (map == AxisMapId::kS_16_24_24) return launch_one<T, 128, Sectioned<16, 24, 24>, kPaged>(p, stream);
    if (map == AxisMapId::kI_22_21_21) return launch_one<T, 128, Interleaved<22, 21, 21>, kPaged>(p, stream);
    if (map == AxisMapId::kI_24_20_20) return launch_one<T, 128, Interleaved<24, 20, 20>, kPaged>(p, stream);
    if (map == AxisMapId::kS_64_0_0) return launch_one<T, 128, Sectioned<64, 0, 0>, kPaged>(p, stream);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_prefill(const PrefillParams &p, prcr_dtype dtype, int head_dim, AxisMapId map,
                          bool paged, hipStream_t stream) {
  if (dtype == PRCR_F32)
    return paged ? dispatch_map<float, true>(p, head_dim, map, stream)
                 : dispatch_map<float, false>(p, head_dim, map, stream);
  return paged ? dispatch_map<uint16_t, true>(p, head_dim, map, stream)
               : dispatch_map<uint16_t, false>(p, head_dim, map, stream);
}

}  // namespace prcr
