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
#include <type_traits>

#include "positions.h"
#include "prcr_internal.h"
#include "rotary.h"

namespace prcr {
namespace {

// Compile-time launch shape, chosen by measurement on MI355X: 4 waves per
// workgroup, 2 row iterations per batch of loads, about 72 rows per wave on large
// problems, non-temporal 16-byte accesses.
#ifndef PRCR_WAVES_PER_BLOCK
#define PRCR_WAVES_PER_BLOCK 4
#endif
#ifndef PRCR_UNROLL
#define PRCR_UNROLL 2
#endif
#ifndef PRCR_ROWS_PER_WAVE
#define PRCR_ROWS_PER_WAVE 72
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
// Logical block of a non-negative slot: one 32-bit division for slots below
// 2^31 (every real cache), the 64-bit one beyond.
__device__ __forceinline__ int64_t block_of(int64_t slot, int32_t block_size) {
  if (slot <= INT32_MAX)
    return static_cast<int64_t>(static_cast<uint32_t>(slot) / static_cast<uint32_t>(block_size));
  return slot / block_size;
}
__device__ __forceinline__ void store16(char *p, u32x4 v) {
#if PRCR_NONTEMPORAL
  store_nt(p, v);
#else
  *reinterpret_cast<u32x4 *>(p) = v;
#endif
}

// One wavefront = one selected token x one run of rows_per_wave (layer, head)
// rows x one array.  The top of the flat workgroup index picks the array: the
// first half rotates and stores keys, the second half copies values.  Workgroups
// are dispatched in index order, so the key half runs before the value half and
// each wave streams one source and one destination (faster than moving both
// arrays in one wave).
//
// Latency.  Vector loads complete in issue order, and a wait for one load also
// waits for every load issued before it, so the wave issues its loads in as few
// dependent rounds as the data allows: (1) its token index, (2) the first rows
// (once the source row is known to be in range) together with every
// per-sequence value, from clamped indices and without branches, and (3) in
// the fused kernel, the coordinates of the sequence's first 64 selected tokens
// (paged: with the destination block-table entry).  Afterwards it always has
// the next batch of rows in flight while it stores the current one.
//
// Key-only memory (v_slot set, no memory values): value waves copy the rows of
// cache slot v_slot[b][m] of the same sequence, which lies below cache_len[b]
// and so is never one of the slots this launch writes.  Their first loads wait
// for that slot (and, paged, its block) instead of being issued early.
//
// kFused (the single-launch revisit): instead of reading new_pos, each key wave
// reduces its sequence's coordinate ranges over the selection (Eq. (8)) with
// wave shuffles and computes its own token's position (Eq. (9)-(10)); the first
// token's wave also writes the sequence's next text position.  The reduction
// costs K_b coordinate reads per wave, which is small at the selection sizes
// the fused path is meant for.
template <typename T, int D, class Map, bool kPaged, int kWaves, int kUnroll, bool kFused>
__global__ __launch_bounds__(kWaves * kWave) void rebind_inject_kernel(const RebindParams p) {
  constexpr int P = D / 2;
  constexpr int E = Store<T>::kPerChunk;   // elements per 16-byte chunk
  constexpr int LPR = P / E;               // lanes per row
  constexpr int RPI = kWave / LPR;         // rows per wave and iteration
  constexpr int kStep = RPI * kUnroll;     // rows per batch of loads
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
  const int64_t n_tblk = (static_cast<int64_t>(p.total_k) + kWaves - 1) / kWaves;
  const int64_t n_work = n_tblk * p.n_row_groups * 2;
  const int64_t L = blockIdx.x;
  // New cache lengths (and, fused, the next position of empty selections),
  // written once by the first workgroup (also when total_k = 0).
  if (L == 0) {
    for (int b = threadIdx.x; b < p.batch; b += blockDim.x) {
      const int kb = p.sel_off[b + 1] - p.sel_off[b];
      if (p.new_cache_len != nullptr) p.new_cache_len[b] = p.cache_len[b] + kb;
      if (kFused && kb == 0) {
        bool nb = false;
        p.next_pos[b] = next_pos_int32(next_text_position(p.mode, p.p_txt[b], 0, false, 0), &nb);
        if (nb && p.err != nullptr) atomicOr(p.err, PRCR_DERR_RANGE);
      }
    }
  }
  if (L >= n_work) return;
  const int64_t tblk = L % n_tblk;
  const int grp = static_cast<int>((L / n_tblk) % p.n_row_groups);
  const bool keys = L < n_tblk * p.n_row_groups;
  const int g = static_cast<int>(tblk * kWaves + wave);
  if (g >= p.total_k) return;
  const int r = lane / LPR;   // this lane's row within an iteration
  const int c = lane % LPR;   // this lane's 16-byte chunk of a half row
  const int rows_total = p.n_layers * p.n_kv_heads;
  const int row0 = grp * p.rows_per_wave;
  const int row_end = min(rows_total, row0 + p.rows_per_wave);

  // The key and value halves of the grid run separate copies of the code below
  // (keys is uniform across the workgroup), so that each half compiles to
  // straight-line loads with no branch on the half between a load and its use.
  auto half = [&](auto key_half) {
    constexpr bool keys = decltype(key_half)::value;
    // Loads that depend only on g are issued first ...
    const int m = p.sel_idx[g];
    double pt = 0.0, ph = 0.0, pw = 0.0;
    if (!kFused && keys) {
      pt = p.new_pos[3 * static_cast<int64_t>(g) + 0];
      ph = p.new_pos[3 * static_cast<int64_t>(g) + 1];
      pw = p.new_pos[3 * static_cast<int64_t>(g) + 2];
    }
    // ... then the sequence of g: (number of offsets <= g) - 1, by a ballot over
    // the offsets held one per lane.  With fewer than 64 sequences one pass holds
    // every offset, and the sequence's own two are read from lanes b and b + 1.
    int cnt = 0, off_lane = 0;
    for (int base = 0; base <= p.batch; base += kWave) {
      const int i = base + lane;
      off_lane = i <= p.batch ? p.sel_off[i] : INT_MAX;
      cnt += __popcll(__ballot(off_lane <= g));
    }
    const int b = __builtin_amdgcn_readfirstlane(cnt - 1);
    const int bq = min(max(b, 0), p.batch - 1);
    int s0, s1;
    if (p.batch < kWave) {
      s0 = __builtin_amdgcn_readfirstlane(__shfl(off_lane, bq));
      s1 = __builtin_amdgcn_readfirstlane(__shfl(off_lane, bq + 1));
    } else {
      s0 = p.sel_off[bq];
      s1 = p.sel_off[bq + 1];
    }
    const bool offsets_ok = b >= 0 && b < p.batch && s0 >= 0 && s0 <= g && g < s1 && s1 <= p.total_k;

    // The source rows exist whenever b and m are in range: start loading them
    // (memory rows; cache rows of a key-only memory are loaded after validation).
    const bool alias_v = !keys && p.v_slot != nullptr;
    const bool src_ok = b >= 0 && b < p.batch && m >= 0 && m < p.max_visual;
    const size_t tok_off = src_ok ? (static_cast<size_t>(b) * p.max_visual + m) * rows_total : 0;
    const char *src = static_cast<const char *>(keys ? p.mem_k : (alias_v ? p.cache_v : p.mem_v)) +
                      (alias_v ? 0 : tok_off * kRowBytes) + c * 16;
    char *dst = static_cast<char *>(keys ? p.cache_k : p.cache_v) + c * 16;
    u32x4 lo[kUnroll], hi[kUnroll];
    if (!alias_v) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = row0 + u * RPI + r;
        if (src_ok && row < row_end) {
          lo[u] = load16(src + static_cast<size_t>(row) * kRowBytes);
          hi[u] = load16(src + static_cast<size_t>(row) * kRowBytes + kHalfBytes);
        }
      }
    }

    // Every per-sequence value is loaded in the same round trip as the rows, from
    // clamped indices (always inside the arrays) and without branches, so that no
    // load waits on another.  The fused kernel also loads the text position, this
    // token's coordinates and the sequence's first 64 selected indices (Eq. (8)).
    const int nvis = p.n_visual[bq];
    const int64_t clen = p.cache_len[bq];
    const int K = s1 - s0;
    int64_t ptxt = 0;
    int cm0 = 0, cm1 = 0, cm2 = 0, mj0 = -1;
    if constexpr (kFused && keys) {
      ptxt = p.p_txt[bq];
      const int mc = min(max(m, 0), p.max_visual - 1);
      const int32_t *cm = p.coords + (static_cast<int64_t>(bq) * p.max_visual + mc) * 3;
      cm0 = cm[0];
      cm1 = cm[1];
      cm2 = cm[2];
      mj0 = p.sel_idx[min(max(s0 + lane, 0), p.total_k - 1)];
    }

    // Validation, without branches: a value used only inside a branch could have
    // its load moved into that branch, a round trip later.
    const int64_t slot = clen + (g - s0);
    const bool index_ok = m >= 0 && m < nvis && m < p.max_visual;
    bool ok = offsets_ok && index_ok;
    int flags = !offsets_ok ? PRCR_DERR_OFFSETS : (index_ok ? 0 : PRCR_DERR_INDEX);
    // Destination slot.  Paged: its block-table entry is read at once, from a
    // clamped logical block (always inside the table); a block beyond the table
    // is flagged below.
    int64_t slot_id = -1, blk = 0, off = 0;
    int slot_flag = 0;
    if constexpr (kPaged) {
      const int64_t lb = slot >= 0 ? block_of(slot, p.block_size) : -1;
      const int64_t lbc = min(max(lb, int64_t{0}), static_cast<int64_t>(p.max_blocks) - 1);
      blk = p.block_table[static_cast<int64_t>(bq) * p.max_blocks + lbc];
      off = slot - lb * p.block_size;
      if (lb < 0 || lb >= p.max_blocks) slot_flag = PRCR_DERR_CAPACITY;
    }
    if constexpr (kFused && keys) {
      // Eq. (8): ranges of the sequence's valid selected coordinates, over a
      // well-formed sequence (a malformed one reduces over nothing).
      // The positions are then formed whatever the validity, so that the values
      // loaded above are used outside any branch: used only inside one, their
      // loads could be moved into it, a round trip later.
      const int Kr = offsets_ok ? K : 0;
      const int lim = min(nvis, p.max_visual);
      const int32_t *cb = p.coords + static_cast<int64_t>(bq) * p.max_visual * 3;
      // The first 64 selected tokens: their coordinates are loaded from a clamped
      // index on every lane, and an absent or invalid entry is masked out.
      const int mc0 = min(max(mj0, 0), p.max_visual - 1);
      const int32_t *cf = cb + 3 * mc0;
      const int f0 = cf[0], f1 = cf[1], f2 = cf[2];
      const bool first = lane < Kr && mj0 >= 0 && mj0 < lim;
      int lo0 = first ? f0 : INT_MAX, lo1 = first ? f1 : INT_MAX, lo2 = first ? f2 : INT_MAX;
      int hi0 = first ? f0 : INT_MIN, hi1 = first ? f1 : INT_MIN, hi2 = first ? f2 : INT_MIN;
      for (int j = lane + kWave; j < Kr; j += kWave) {
        const int mj = p.sel_idx[s0 + j];
        if (mj >= 0 && mj < lim) {
          const int c0 = cb[3 * mj], c1 = cb[3 * mj + 1], c2 = cb[3 * mj + 2];
          lo0 = min(lo0, c0); hi0 = max(hi0, c0);
          lo1 = min(lo1, c1); hi1 = max(hi1, c1);
          lo2 = min(lo2, c2); hi2 = max(hi2, c2);
        }
      }
      for (int o = kWave / 2; o > 0; o >>= 1) {
        lo0 = min(lo0, __shfl_xor(lo0, o)); hi0 = max(hi0, __shfl_xor(hi0, o));
        lo1 = min(lo1, __shfl_xor(lo1, o)); hi1 = max(hi1, __shfl_xor(hi1, o));
        lo2 = min(lo2, __shfl_xor(lo2, o)); hi2 = max(hi2, __shfl_xor(hi2, o));
      }
      // Eq. (9)-(10).  Safe on any input (magnitudes are checked before the
      // integer products); the values only count for a valid token.
      bool range_bad = false;
      const int64_t j = static_cast<int64_t>(g) - s0;
      pt = reassigned(p.mode, ptxt, p.l_ext, K, j, lo0, hi0, cm0, &range_bad);
      ph = reassigned(p.mode, ptxt, p.l_ext, K, j, lo1, hi1, cm1, &range_bad);
      pw = reassigned(p.mode, ptxt, p.l_ext, K, j, lo2, hi2, cm2, &range_bad);
      if (!ok) pt = ph = pw = __builtin_nan("");
      if (offsets_ok && grp == 0 && lane == 0) {
        if (p.pos_out != nullptr) {
          p.pos_out[3 * static_cast<int64_t>(g) + 0] = pt;
          p.pos_out[3 * static_cast<int64_t>(g) + 1] = ph;
          p.pos_out[3 * static_cast<int64_t>(g) + 2] = pw;
        }
        if (g == s0) {
          const bool any_valid = lo0 <= hi0;
          const int64_t span = any_valid ? max(static_cast<int64_t>(hi0) - lo0,
                                               max(static_cast<int64_t>(hi1) - lo1,
                                                   static_cast<int64_t>(hi2) - lo2))
                                         : 0;
          bool next_bad = false;
          p.next_pos[b] = next_pos_int32(next_text_position(p.mode, ptxt, K, any_valid, span),
                                         &next_bad);
          if (next_bad && p.err != nullptr) atomicOr(p.err, PRCR_DERR_RANGE);
        }
        if (ok && range_bad && p.err != nullptr) atomicOr(p.err, PRCR_DERR_RANGE);
      }
    }
    // Key-only memory: the value slot must be one of the sequence's filled slots.
    int64_t vslot = 0, vpool = 0;
    if (ok && p.v_slot != nullptr) {
      vslot = p.v_slot[static_cast<int64_t>(b) * p.max_visual + m];
      if (vslot < 0 || vslot >= clen) {
        ok = false;
        flags = PRCR_DERR_INDEX;
      } else if constexpr (kPaged) {
        const int64_t lb = block_of(vslot, p.block_size);
        if (lb >= p.max_blocks) {
          ok = false;
          flags = PRCR_DERR_CAPACITY;
        } else {
          const int64_t vb = p.block_table[static_cast<int64_t>(b) * p.max_blocks + lb];
          if (vb < 0 || vb >= p.n_blocks) {
            ok = false;
            flags = PRCR_DERR_BLOCK;
          } else {
            vpool = vb * p.block_size + (vslot - lb * p.block_size);
          }
        }
      } else if (vslot >= p.s_max) {
        ok = false;
        flags = PRCR_DERR_CAPACITY;
      }
    }
    if (ok) {
      if constexpr (kPaged) {
        if (slot_flag != 0) {
          ok = false;
          flags = slot_flag;
        } else if (blk < 0 || blk >= p.n_blocks) {
          ok = false;
          flags = PRCR_DERR_BLOCK;
        } else {
          slot_id = blk * p.block_size + off;
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

    // Destination slot within a layer's block pool (paged only).
    const size_t dst_pool = kPaged ? static_cast<size_t>(blk) * p.block_size + off : 0;
    // Byte offset of (layer, head) row `row` of a cache slot: `pool` is the slot
    // within a layer's block pool (paged), `sl` the sequence's slot (contiguous).
    auto cache_offset = [&](int row, size_t pool, int64_t sl) -> size_t {
      if constexpr (kPaged) {
        const int l = row / p.n_kv_heads;
        const int h = row - l * p.n_kv_heads;
        return ((static_cast<size_t>(l) * p.n_blocks * p.block_size + pool) * p.n_kv_heads + h) *
               kRowBytes;
      } else {
        return ((static_cast<size_t>(b) * rows_total + row) * p.s_max + sl) * kRowBytes;
      }
    };
    auto dst_offset = [&](int row) -> size_t { return cache_offset(row, dst_pool, slot); };
    auto src_offset = [&](int row) -> size_t {
      return alias_v ? cache_offset(row, static_cast<size_t>(vpool), vslot)
                     : static_cast<size_t>(row) * kRowBytes;
    };
    if (alias_v) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = row0 + u * RPI + r;
        if (row < row_end) {
          lo[u] = load16(src + src_offset(row));
          hi[u] = load16(src + src_offset(row) + kHalfBytes);
        }
      }
    }

    // cos/sin of this token's angles (keys only): lane i computes pair i (mod P),
    // then lane (r, c) gathers the pairs c*E .. c*E+E-1 of its two chunks.
    double cs[E], sn[E];
    if (keys) {
      const int pair = lane % P;
      const int ax = Map::axis(pair);
      double sv, cv;
      sincos((ax == 0 ? pt : (ax == 1 ? ph : pw)) * p.inv_freq[pair], &sv, &cv);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        cs[e] = __shfl(cv, c * E + e);
        sn[e] = __shfl(sv, c * E + e);
      }
    }

    // Rows rb .. rb + kStep - 1 of the batch held in lo/hi: rotated (keys) and
    // stored.
    auto store_batch = [&](int rb) {
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = rb + u * RPI + r;
        if (row < row_end) {
          u32x4 ol = lo[u], oh = hi[u];
          if (keys) Store<T>::rotate(lo[u], hi[u], cs, sn, ol, oh);
          const size_t d = dst_offset(row);
          store16(dst + d, ol);
          store16(dst + d + kHalfBytes, oh);
        }
      }
    };
    // The next batch is in flight while this one is stored.  Its loads are
    // issued unconditionally (rows past the run reload its last row), so that
    // the wait before the stores covers exactly this batch; the last batch,
    // which has no next one, is stored after the loop.
    int rb = row0;
    for (; rb + kStep < row_end; rb += kStep) {
      u32x4 nlo[kUnroll], nhi[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int row = min(rb + kStep + u * RPI + r, row_end - 1);
        nlo[u] = load16(src + src_offset(row));
        nhi[u] = load16(src + src_offset(row) + kHalfBytes);
      }
      store_batch(rb);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        lo[u] = nlo[u];
        hi[u] = nhi[u];
      }
    }
    store_batch(rb);
  };
  if (keys)
    half(std::true_type{});
  else
    half(std::false_type{});
}

constexpr int kWavesPerBlock = PRCR_WAVES_PER_BLOCK;
constexpr int kUnrollRows = PRCR_UNROLL;

template <typename T, int D, class Map, bool kPaged, bool kFused>
hipError_t launch_one(const RebindParams &in, hipStream_t stream) {
  constexpr int P = D / 2;
  constexpr int LPR = P / Store<T>::kPerChunk;
  constexpr int RPI = kWave / LPR;
  constexpr int kStep = RPI * kUnrollRows;
  RebindParams p = in;
  // Rows of one token handled by one wave: a whole number of load batches.
  // Large problems use about PRCR_ROWS_PER_WAVE rows per wave; small ones are
  // spread over at least kMinWaves waves per array (down to one batch per wave)
  // so that their latency is a few load round trips.
  constexpr int64_t kMinWaves = 4096;
  const int rows_total = p.n_layers * p.n_kv_heads;
  const int64_t rows_all = static_cast<int64_t>(p.total_k) * rows_total;
  int64_t target = PRCR_ROWS_PER_WAVE;
  if (rows_all < target * kMinWaves) target = rows_all / kMinWaves;
  target = (target + kStep - 1) / kStep * kStep;
  if (target < kStep) target = kStep;
  const int64_t groups = (rows_total + target - 1) / target;
  int64_t per = (rows_total + groups - 1) / groups;
  per = (per + kStep - 1) / kStep * kStep;
  p.rows_per_wave = static_cast<int32_t>(per);
  p.n_row_groups = static_cast<int32_t>((rows_total + per - 1) / per);
  if (p.n_row_groups > 65535) return hipErrorInvalidConfiguration;
  // One flat grid over (token block, row group, K|V); at least one workgroup so
  // that the new cache lengths are written when nothing is selected.
  const int64_t n_tblk = (static_cast<int64_t>(p.total_k) + kWavesPerBlock - 1) / kWavesPerBlock;
  int64_t n_work = n_tblk * p.n_row_groups * 2;
  if (n_work < 1) n_work = 1;
  if (!grid_fits(n_work, kWavesPerBlock * kWave)) return hipErrorInvalidConfiguration;
  const dim3 grid(static_cast<unsigned>(n_work));
  rebind_inject_kernel<T, D, Map, kPaged, kWavesPerBlock, kUnrollRows, kFused>
      <<<grid, kWavesPerBlock * kWave, 0, stream>>>(p);
  return hipGetLastError();
}

template <typename T, bool kPaged, bool kFused>
hipError_t dispatch_map(const RebindParams &p, int head_dim, AxisMapId map, hipStream_t stream) {
  if (head_dim == 64) {
    if (map == AxisMapId::kS_8_12_12)
      return launch_one<T, 64, Sectioned<8, 12, 12>, kPaged, kFused>(p, stream);
    if (map == AxisMapId::kI_11_11_10)
      return launch_one<T, 64, Interleaved<11, 11, 10>, kPaged, kFused>(p, stream);
    if (map == AxisMapId::kS_32_0_0)
      return launch_one<T, 64, Sectioned<32, 0, 0>, kPaged, kFused>(p, stream);
  } else if (head_dim == 128) {
    if (map == AxisMapId::kS_16_24_24)
      return launch_one<T, 128, Sectioned<16, 24, 24>, kPaged, kFused>(p, stream);
    if (map == AxisMapId::kI_22_21_21)
      return launch_one<T, 128, Interleaved<22, 21, 21>, kPaged, kFused>(p, stream);
    if (map == AxisMapId::kI_24_20_20)
      return launch_one<T, 128, Interleaved<24, 20, 20>, kPaged, kFused>(p, stream);
    if (map == AxisMapId::kS_64_0_0)
      return launch_one<T, 128, Sectioned<64, 0, 0>, kPaged, kFused>(p, stream);
  }
  return hipErrorInvalidValue;
}

template <typename T>
hipError_t dispatch_layout(const RebindParams &p, int head_dim, AxisMapId map, bool paged,
                           bool fused, hipStream_t stream) {
  if (paged)
    return fused ? dispatch_map<T, true, true>(p, head_dim, map, stream)
                 : dispatch_map<T, true, false>(p, head_dim, map, stream);
  return fused ? dispatch_map<T, false, true>(p, head_dim, map, stream)
               : dispatch_map<T, false, false>(p, head_dim, map, stream);
}

}  // namespace

hipError_t launch_rebind(const RebindParams &p, prcr_dtype dtype, int head_dim, AxisMapId map,
                         bool paged, bool fused, hipStream_t stream) {
  if (dtype == PRCR_F32) return dispatch_layout<float>(p, head_dim, map, paged, fused, stream);
  return dispatch_layout<uint16_t>(p, head_dim, map, paged, fused, stream);
}

}  // namespace prcr
