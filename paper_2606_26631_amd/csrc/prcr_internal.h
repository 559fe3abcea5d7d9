// Internal declarations shared by the host API and the HIP kernel translation
// units.  Not part of the public ABI.
#pragma once

#include <cstddef>
#include <cstdint>

#include <hip/hip_runtime.h>

#include "prcr.h"

namespace prcr {

constexpr int kMaxPairs = 64;        // head_dim <= 128
constexpr int kWave = 64;            // CDNA wavefront width

// ---------------------------------------------------------------------------
// Rotary axis maps, resolved at compile time.  Pair i takes its position from
// axis(i): 0 = t, 1 = h, 2 = w.
// ---------------------------------------------------------------------------
template <int ST, int SH, int SW>
struct Sectioned {
  static constexpr int kPairs = ST + SH + SW;
  __host__ __device__ static constexpr int axis(int i) {
    return i < ST ? 0 : (i < ST + SH ? 1 : 2);
  }
};

template <int ST, int SH, int SW>
struct Interleaved {
  static constexpr int kPairs = ST + SH + SW;
  __host__ __device__ static constexpr int axis(int i) {
    return (i % 3 == 1 && i < 3 * SH) ? 1 : ((i % 3 == 2 && i < 3 * SW) ? 2 : 0);
  }
};

// ---------------------------------------------------------------------------
// Kernel parameter blocks (passed by value as kernel arguments).
// ---------------------------------------------------------------------------
struct ReassignParams {
  const int32_t *coords;
  const int32_t *n_visual;
  const int32_t *sel_off;
  const int32_t *sel_idx;
  const int32_t *p_txt;
  double *new_pos;
  int32_t *next_pos;
  int32_t *err;
  int32_t batch, max_visual, total_k, mode, l_ext;
};

struct RebindParams {
  const void *mem_k;
  const void *mem_v;              // null for a key-only memory
  const int32_t *v_slot;          // key-only memory: [batch][max_visual] cache slot of the values
  const int32_t *n_visual;
  const int32_t *sel_off;
  const int32_t *sel_idx;
  const double *new_pos;
  void *cache_k;
  void *cache_v;
  const int32_t *block_table;
  const int32_t *cache_len;
  int32_t *new_cache_len;
  int64_t *slot_mapping;
  int32_t *err;
  int32_t batch, max_visual, n_layers, n_kv_heads, total_k;
  int32_t s_max, block_size, max_blocks, n_blocks;
  int32_t rows_per_wave;          // rows (layer, head) of one token handled by one wave
  int32_t n_row_groups;           // ceil(n_layers * n_kv_heads / rows_per_wave)
  // Fused revisit only (positions computed in the kernel instead of read):
  const int32_t *coords;          // [batch][max_visual][3]
  const int32_t *p_txt;           // [batch]
  double *pos_out;                // [total_k][3] or null
  int32_t *next_pos;              // [batch]
  int32_t mode, l_ext;
  double inv_freq[kMaxPairs];     // theta^(-2i/head_dim)
};

struct StoreParams {
  void *mem_k;
  void *mem_v;
  const int32_t *n_visual;
  const void *raw_k;
  const void *raw_v;
  const int32_t *vis_rows;
  int32_t *err;
  int32_t batch, max_visual, n_layers, n_kv_heads, layer, s_src;
  int32_t row_bytes;              // n_kv_heads * head_dim * element size
};

struct PrefillParams {
  const void *raw_k;
  const void *raw_v;
  const int32_t *pos;             // [batch][s_src][3] position ids
  const int32_t *n_tokens;        // [batch]
  const int32_t *vis_index;       // [batch][s_src], -1 for non-visual rows
  void *mem_k;
  void *mem_v;                    // null for a key-only memory
  int32_t *v_slot;                // key-only memory: out [batch][max_visual], or null
  int32_t *coords;
  const int32_t *n_visual;
  void *cache_k;
  void *cache_v;
  const int32_t *block_table;
  const int32_t *cache_start;     // [batch]
  int32_t *err;
  int32_t batch, s_src, max_visual, n_layers, n_kv_heads, layer, write_coords;
  int32_t s_max, block_size, max_blocks, n_blocks;
  double inv_freq[kMaxPairs];
};

struct DecodeParams {
  const void *q;                  // [batch][n_q_heads][head_dim]
  const int32_t *q_pos;           // [batch]
  const int32_t *cache_len;       // [batch]
  const void *cache_k;
  const void *cache_v;
  const int32_t *block_table;
  float *out;                     // [batch][n_q_heads][head_dim]
  float *ws;                      // [batch][n_q_heads][n_split][head_dim + 2]
  int32_t *err;
  int32_t batch, n_layers, n_kv_heads, n_q_heads, layer;
  int32_t s_max, block_size, max_blocks, n_blocks;
  int32_t block_shift;            // log2(block_size) if a power of two, else -1
  int32_t n_split;                // workgroups per (sequence, KV head)
  float scale;
  double inv_freq[kMaxPairs];
};

// Axis-map identifiers understood by the dispatcher.
enum class AxisMapId : int {
  kS_8_12_12 = 0,
  kI_11_11_10 = 1,
  kS_16_24_24 = 2,
  kI_22_21_21 = 3,
  kI_24_20_20 = 4,
  kS_32_0_0 = 5,     // 1-D rotary, head_dim 64: every pair on the t axis
  kS_64_0_0 = 6,     // 1-D rotary, head_dim 128
  kUnsupported = -1,
};

AxisMapId axis_map_id(const prcr_rope &rope);

// The dispatch packet holds each grid dimension as a 32-bit count of work-items:
// a launcher refuses (hipErrorInvalidConfiguration, before any HIP call) a grid
// whose x extent would not fit.
inline bool grid_fits(int64_t blocks, int threads) {
  return blocks >= 1 && blocks <= static_cast<int64_t>(UINT32_MAX) / threads;
}
int axis_of_pair(AxisMapId id, int i);

// Launchers (return the hipError_t of the launch).
hipError_t launch_reassign(const ReassignParams &p, hipStream_t stream);
hipError_t launch_rebind(const RebindParams &p, prcr_dtype dtype, int head_dim, AxisMapId map,
                         bool paged, bool fused, hipStream_t stream);
hipError_t launch_store(const StoreParams &p, hipStream_t stream);
hipError_t launch_prefill(const PrefillParams &p, prcr_dtype dtype, int head_dim, AxisMapId map,
                          bool paged, hipStream_t stream);
hipError_t launch_decode(const DecodeParams &p, prcr_dtype dtype, int head_dim, bool paged,
                         hipStream_t stream);
int decode_splits(int64_t capacity, int batch, int n_kv_heads, int group);

// A launcher's own refusal of a grid too large for one dispatch is a size error
// found before any HIP call (PRCR_ERR_SHAPE); anything else the runtime reports
// is a launch error (PRCR_ERR_HIP).
prcr_status launch_status(hipError_t e);

// Host checks and parameter block shared by the decode entry points: everything
// but the split-K workspace pointer, whose byte size is returned in *ws_bytes.
prcr_status prepare_decode(const prcr_rope *rope, const prcr_cache *cache, prcr_dtype dtype,
                           int32_t batch, int32_t n_layers, int32_t n_kv_heads, int32_t layer,
                           const void *q, int32_t n_q_heads, const int32_t *q_pos,
                           const int32_t *cache_len, float scale, float *out, int32_t *err_flag,
                           DecodeParams *out_params, size_t *ws_bytes);

}  // namespace prcr
