// extern "C" entry points: structural validation on the host, then one kernel
// launch on the caller's stream.  No entry point allocates or keeps state.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <cstddef>

#include "prcr_internal.h"

using namespace prcr;

namespace {

constexpr int32_t kVersion = 1 * 10000 + 3 * 100 + 2;
constexpr int64_t kMaxDecodeSlots = int64_t{1} << 30;   // decode: cache capacity per sequence

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int elem_bytes(prcr_dtype d) { return d == PRCR_F32 ? 4 : 2; }

// A launcher's own refusal of a grid too large for one dispatch is a size error
// found before any HIP call; anything else the runtime reports is a launch error.
prcr_status launch_status(hipError_t e) {
  if (e == hipSuccess) return PRCR_OK;
  return e == hipErrorInvalidConfiguration ? PRCR_ERR_SHAPE : PRCR_ERR_HIP;
}

prcr_status check_rope(const prcr_rope *rope) {
  if (rope == nullptr) return PRCR_ERR_NULL;
  const int d = rope->head_dim;
  if (d < 2 || d % 2 != 0 || d / 2 > kMaxPairs) return PRCR_ERR_SHAPE;
  if (rope->section[0] < 0 || rope->section[1] < 0 || rope->section[2] < 0) return PRCR_ERR_SHAPE;
  if (static_cast<int64_t>(rope->section[0]) + rope->section[1] + rope->section[2] != d / 2)
    return PRCR_ERR_SHAPE;
  if (rope->interleaved != 0 && rope->interleaved != 1) return PRCR_ERR_SHAPE;
  if (!(rope->theta > 0.0) || !std::isfinite(rope->theta)) return PRCR_ERR_SHAPE;
  return PRCR_OK;
}

prcr_status check_mem(const prcr_mem *mem, bool need_coords) {
  if (mem == nullptr || mem->k == nullptr || mem->n_visual == nullptr) return PRCR_ERR_NULL;
  // A key-only memory names the cache slot of each value row instead.
  if (mem->v == nullptr && mem->v_slot == nullptr) return PRCR_ERR_NULL;
  if (need_coords && mem->coords == nullptr) return PRCR_ERR_NULL;
  if (mem->dtype != PRCR_F32 && mem->dtype != PRCR_BF16) return PRCR_ERR_DTYPE;
  if (mem->batch < 1 || mem->max_visual < 1 || mem->n_layers < 1 || mem->n_kv_heads < 1)
    return PRCR_ERR_SHAPE;
  const int d = mem->head_dim;
  if (d < 2 || d % 2 != 0 || d / 2 > kMaxPairs) return PRCR_ERR_SHAPE;
  // Each half row must be a whole number of 16-byte chunks.
  if ((d / 2) * elem_bytes(mem->dtype) % 16 != 0) return PRCR_ERR_SHAPE;
  if (static_cast<int64_t>(mem->n_layers) * mem->n_kv_heads > INT32_MAX / 2) return PRCR_ERR_SHAPE;
  // One layer's rows of a token (all KV heads) must have a 32-bit byte size.
  if (static_cast<int64_t>(mem->n_kv_heads) * d * elem_bytes(mem->dtype) > INT32_MAX) return PRCR_ERR_SHAPE;
  if (!aligned(mem->k, 16) || !aligned(mem->v, 16) || !aligned(mem->n_visual, 4))
    return PRCR_ERR_ALIGN;
  if (mem->v == nullptr && !aligned(mem->v_slot, 4)) return PRCR_ERR_ALIGN;
  if (need_coords && !aligned(mem->coords, 4)) return PRCR_ERR_ALIGN;
  return PRCR_OK;
}

prcr_status check_selection(const prcr_mem *mem, const int32_t *sel_off, const int32_t *sel_idx,
                            int32_t total_k) {
  if (sel_off == nullptr) return PRCR_ERR_NULL;
  if (total_k < 0) return PRCR_ERR_SHAPE;
  if (total_k > 0 && sel_idx == nullptr) return PRCR_ERR_NULL;
  if (!aligned(sel_off, 4) || (sel_idx != nullptr && !aligned(sel_idx, 4))) return PRCR_ERR_ALIGN;
  (void)mem;
  return PRCR_OK;
}

// The cache descriptor every entry point that touches a cache validates: layout
// flag, pointers, geometry, alignment.
prcr_status check_cache(const prcr_cache *cache) {
  if (cache == nullptr || cache->k == nullptr || cache->v == nullptr) return PRCR_ERR_NULL;
  if (cache->paged != 0 && cache->paged != 1) return PRCR_ERR_SHAPE;
  if (cache->paged) {
    if (cache->block_table == nullptr) return PRCR_ERR_NULL;
    if (cache->block_size < 1 || cache->max_blocks < 1 || cache->n_blocks < 1) return PRCR_ERR_SHAPE;
    if (!aligned(cache->block_table, 4)) return PRCR_ERR_ALIGN;
  } else if (cache->s_max < 1) {
    return PRCR_ERR_SHAPE;
  }
  if (!aligned(cache->k, 16) || !aligned(cache->v, 16)) return PRCR_ERR_ALIGN;
  return PRCR_OK;
}

}  // namespace

extern "C" {

const char *prcr_status_str(prcr_status s) {
  switch (s) {
    case PRCR_OK: return "ok";
    case PRCR_ERR_NULL: return "a required pointer is NULL";
    case PRCR_ERR_SHAPE: return "a size or count is out of range or inconsistent";
    case PRCR_ERR_DTYPE: return "unknown element type";
    case PRCR_ERR_ALIGN: return "a pointer is not aligned as required";
    case PRCR_ERR_MODE: return "unknown reassignment mode or negative l_ext";
    case PRCR_ERR_UNSUPPORTED: return "no compiled kernel for this head_dim / axis map";
    case PRCR_ERR_ALIAS: return "an output aliases an input it must not alias";
    case PRCR_ERR_HIP: return "HIP launch error";
  }
  return "unknown status";
}

int32_t prcr_version(void) { return kVersion; }

prcr_status prcr_inv_freq(const prcr_rope *rope, double *out_host) {
  const prcr_status st = check_rope(rope);
  if (st != PRCR_OK) return st;
  if (out_host == nullptr) return PRCR_ERR_NULL;
  for (int i = 0; i < rope->head_dim / 2; ++i)
    out_host[i] = std::pow(rope->theta, -(2.0 * i) / rope->head_dim);
  return PRCR_OK;
}

prcr_status prcr_pair_axis(const prcr_rope *rope, int32_t *out_host) {
  const prcr_status st = check_rope(rope);
  if (st != PRCR_OK) return st;
  if (out_host == nullptr) return PRCR_ERR_NULL;
  const AxisMapId id = axis_map_id(*rope);
  if (id == AxisMapId::kUnsupported) return PRCR_ERR_UNSUPPORTED;
  for (int i = 0; i < rope->head_dim / 2; ++i) out_host[i] = axis_of_pair(id, i);
  return PRCR_OK;
}

prcr_status prcr_store_raw(const prcr_mem *mem, int32_t layer, const void *raw_k, const void *raw_v,
                           int32_t s_src, const int32_t *vis_rows, int32_t *err_flag,
                           hipStream_t stream) {
  prcr_status st = check_mem(mem, false);
  if (st != PRCR_OK) return st;
  if (raw_k == nullptr || (mem->v != nullptr && raw_v == nullptr) || vis_rows == nullptr)
    return PRCR_ERR_NULL;
  if (layer < 0 || layer >= mem->n_layers || s_src < 1 || mem->batch > 65535) return PRCR_ERR_SHAPE;
  if (!aligned(raw_k, 16) || !aligned(raw_v, 16) || !aligned(vis_rows, 4) ||
      (err_flag != nullptr && !aligned(err_flag, 4)))
    return PRCR_ERR_ALIGN;
  StoreParams p{};
  p.mem_k = mem->k;
  p.mem_v = mem->v;
  p.n_visual = mem->n_visual;
  p.raw_k = raw_k;
  p.raw_v = mem->v != nullptr ? raw_v : nullptr;
  p.vis_rows = vis_rows;
  p.err = err_flag;
  p.batch = mem->batch;
  p.max_visual = mem->max_visual;
  p.n_layers = mem->n_layers;
  p.n_kv_heads = mem->n_kv_heads;
  p.layer = layer;
  p.s_src = s_src;
  p.row_bytes = mem->n_kv_heads * mem->head_dim * elem_bytes(mem->dtype);
  return launch_status(launch_store(p, stream));
}

prcr_status prcr_reassign_coords(const prcr_mem *mem, const int32_t *sel_off, const int32_t *sel_idx,
                                 int32_t total_k, const int32_t *p_txt, prcr_mode mode, int32_t l_ext,
                                 double *new_pos, int32_t *next_pos, int32_t *err_flag,
                                 hipStream_t stream) {
  prcr_status st = check_mem(mem, true);
  if (st != PRCR_OK) return st;
  st = check_selection(mem, sel_off, sel_idx, total_k);
  if (st != PRCR_OK) return st;
  if (p_txt == nullptr || next_pos == nullptr) return PRCR_ERR_NULL;
  if (total_k > 0 && new_pos == nullptr) return PRCR_ERR_NULL;
  if (mode < PRCR_MODE_PCR || mode > PRCR_MODE_PCR_RIGHT || l_ext < 0) return PRCR_ERR_MODE;
  if (!aligned(p_txt, 4) || !aligned(next_pos, 4) || (new_pos != nullptr && !aligned(new_pos, 8)) ||
      (err_flag != nullptr && !aligned(err_flag, 4)))
    return PRCR_ERR_ALIGN;
  ReassignParams p{};
  p.coords = mem->coords;
  p.n_visual = mem->n_visual;
  p.sel_off = sel_off;
  p.sel_idx = sel_idx;
  p.p_txt = p_txt;
  p.new_pos = new_pos;
  p.next_pos = next_pos;
  p.err = err_flag;
  p.batch = mem->batch;
  p.max_visual = mem->max_visual;
  p.total_k = total_k;
  p.mode = static_cast<int32_t>(mode);
  p.l_ext = l_ext;
  return launch_status(launch_reassign(p, stream));
}

}  // extern "C"

namespace {

// Shared checks and parameter block of prcr_rebind_inject and prcr_revisit.
prcr_status prepare_rebind(const prcr_rope *rope, const prcr_mem *mem, const int32_t *sel_off,
                           const int32_t *sel_idx, int32_t total_k, const prcr_cache *cache,
                           const int32_t *cache_len, int32_t *new_cache_len, int64_t *slot_mapping,
                           int32_t *err_flag, bool need_coords, RebindParams *out, AxisMapId *map) {
  prcr_status st = check_rope(rope);
  if (st != PRCR_OK) return st;
  st = check_mem(mem, need_coords);
  if (st != PRCR_OK) return st;
  if (rope->head_dim != mem->head_dim) return PRCR_ERR_SHAPE;
  st = check_selection(mem, sel_off, sel_idx, total_k);
  if (st != PRCR_OK) return st;
  st = check_cache(cache);
  if (st != PRCR_OK) return st;
  if (cache_len == nullptr) return PRCR_ERR_NULL;
  if (!aligned(cache_len, 4) ||
      (new_cache_len != nullptr && !aligned(new_cache_len, 4)) ||
      (slot_mapping != nullptr && !aligned(slot_mapping, 8)) ||
      (err_flag != nullptr && !aligned(err_flag, 4)))
    return PRCR_ERR_ALIGN;
  if (new_cache_len != nullptr && new_cache_len == cache_len) return PRCR_ERR_ALIAS;
  *map = axis_map_id(*rope);
  if (*map == AxisMapId::kUnsupported) return PRCR_ERR_UNSUPPORTED;

  RebindParams &p = *out;
  p = RebindParams{};
  p.mem_k = mem->k;
  p.mem_v = mem->v;
  p.v_slot = mem->v == nullptr ? mem->v_slot : nullptr;
  p.n_visual = mem->n_visual;
  p.sel_off = sel_off;
  p.sel_idx = sel_idx;
  p.cache_k = cache->k;
  p.cache_v = cache->v;
  p.block_table = cache->block_table;
  p.cache_len = cache_len;
  p.new_cache_len = new_cache_len;
  p.slot_mapping = slot_mapping;
  p.err = err_flag;
  p.batch = mem->batch;
  p.max_visual = mem->max_visual;
  p.n_layers = mem->n_layers;
  p.n_kv_heads = mem->n_kv_heads;
  p.total_k = total_k;
  p.s_max = cache->s_max;
  p.block_size = cache->block_size;
  p.max_blocks = cache->max_blocks;
  p.n_blocks = cache->n_blocks;
  for (int i = 0; i < rope->head_dim / 2; ++i)
    p.inv_freq[i] = std::pow(rope->theta, -(2.0 * i) / rope->head_dim);
  return PRCR_OK;
}

}  // namespace

extern "C" {

prcr_status prcr_rebind_inject(const prcr_rope *rope, const prcr_mem *mem, const int32_t *sel_off,
                               const int32_t *sel_idx, int32_t total_k, const double *new_pos,
                               const prcr_cache *cache, const int32_t *cache_len,
                               int32_t *new_cache_len, int64_t *slot_mapping, int32_t *err_flag,
                               hipStream_t stream) {
  RebindParams p;
  AxisMapId map;
  const prcr_status st = prepare_rebind(rope, mem, sel_off, sel_idx, total_k, cache, cache_len,
                                        new_cache_len, slot_mapping, err_flag, false, &p, &map);
  if (st != PRCR_OK) return st;
  if (total_k > 0 && new_pos == nullptr) return PRCR_ERR_NULL;
  if (new_pos != nullptr && !aligned(new_pos, 8)) return PRCR_ERR_ALIGN;
  p.new_pos = new_pos;
  const hipError_t e = launch_rebind(p, mem->dtype, mem->head_dim, map, cache->paged != 0, false, stream);
  return launch_status(e);
}

prcr_status prcr_prefill_capture(const prcr_rope *rope, const prcr_mem *mem, int32_t layer,
                                 const void *raw_k, const void *raw_v, int32_t s_src,
                                 const int32_t *pos, const int32_t *n_tokens,
                                 const int32_t *vis_index, int32_t write_coords,
                                 const prcr_cache *cache, const int32_t *cache_start,
                                 int32_t *err_flag, hipStream_t stream) {
  prcr_status st = check_rope(rope);
  if (st != PRCR_OK) return st;
  st = check_mem(mem, write_coords != 0);
  if (st != PRCR_OK) return st;
  if (rope->head_dim != mem->head_dim) return PRCR_ERR_SHAPE;
  if (raw_k == nullptr || raw_v == nullptr || pos == nullptr || n_tokens == nullptr ||
      vis_index == nullptr || cache_start == nullptr)
    return PRCR_ERR_NULL;
  st = check_cache(cache);
  if (st != PRCR_OK) return st;
  if (layer < 0 || layer >= mem->n_layers || s_src < 1) return PRCR_ERR_SHAPE;
  if (!aligned(raw_k, 16) || !aligned(raw_v, 16) || !aligned(pos, 4) || !aligned(n_tokens, 4) ||
      !aligned(vis_index, 4) || !aligned(cache_start, 4) ||
      (err_flag != nullptr && !aligned(err_flag, 4)))
    return PRCR_ERR_ALIGN;
  const AxisMapId map = axis_map_id(*rope);
  if (map == AxisMapId::kUnsupported) return PRCR_ERR_UNSUPPORTED;
  PrefillParams p{};
  p.raw_k = raw_k;
  p.raw_v = raw_v;
  p.pos = pos;
  p.n_tokens = n_tokens;
  p.vis_index = vis_index;
  p.mem_k = mem->k;
  p.mem_v = mem->v;
  p.v_slot = mem->v == nullptr ? mem->v_slot : nullptr;
  p.coords = mem->coords;
  p.n_visual = mem->n_visual;
  p.cache_k = cache->k;
  p.cache_v = cache->v;
  p.block_table = cache->block_table;
  p.cache_start = cache_start;
  p.err = err_flag;
  p.batch = mem->batch;
  p.s_src = s_src;
  p.max_visual = mem->max_visual;
  p.n_layers = mem->n_layers;
  p.n_kv_heads = mem->n_kv_heads;
  p.layer = layer;
  p.write_coords = write_coords != 0;
  p.s_max = cache->s_max;
  p.block_size = cache->block_size;
  p.max_blocks = cache->max_blocks;
  p.n_blocks = cache->n_blocks;
  for (int i = 0; i < rope->head_dim / 2; ++i)
    p.inv_freq[i] = std::pow(rope->theta, -(2.0 * i) / rope->head_dim);
  const hipError_t e = launch_prefill(p, mem->dtype, mem->head_dim, map, cache->paged != 0, stream);
  return launch_status(e);
}

static prcr_status decode_shape(const prcr_cache *cache, int32_t batch, int32_t n_q_heads,
                               int32_t n_kv_heads, int32_t head_dim, int *n_split) {
  if (cache == nullptr) return PRCR_ERR_NULL;
  if (batch < 1 || batch > 65535 || n_kv_heads < 1 || n_kv_heads > 65535 || n_q_heads < 1 ||
      n_q_heads % n_kv_heads != 0 || n_q_heads / n_kv_heads > 8 || n_q_heads > 65535)
    return PRCR_ERR_SHAPE;
  if (head_dim != 64 && head_dim != 128) return PRCR_ERR_UNSUPPORTED;
  if (cache->paged != 0 && cache->paged != 1) return PRCR_ERR_SHAPE;
  int64_t cap;
  if (cache->paged) {
    if (cache->block_size < 1 || cache->max_blocks < 1 || cache->n_blocks < 1) return PRCR_ERR_SHAPE;
    cap = static_cast<int64_t>(cache->max_blocks) * cache->block_size;
  } else {
    if (cache->s_max < 1) return PRCR_ERR_SHAPE;
    cap = cache->s_max;
  }
  // Slot indices, plus a few batches of look-ahead, stay far inside 32 bits.
  if (cap > kMaxDecodeSlots) return PRCR_ERR_SHAPE;
  *n_split = decode_splits(cap, batch, n_kv_heads);
  return PRCR_OK;
}

prcr_status prcr_decode_workspace_size(const prcr_cache *cache, int32_t batch, int32_t n_q_heads,
                                       int32_t n_kv_heads, int32_t head_dim, size_t *bytes) {
  if (bytes == nullptr) return PRCR_ERR_NULL;
  int n_split = 0;
  const prcr_status st = decode_shape(cache, batch, n_q_heads, n_kv_heads, head_dim, &n_split);
  if (st != PRCR_OK) return st;
  *bytes = static_cast<size_t>(batch) * n_q_heads * n_split * (head_dim + 2) * sizeof(float);
  return PRCR_OK;
}

prcr_status prcr_decode_attention(const prcr_rope *rope, const prcr_cache *cache, prcr_dtype dtype,
                                  int32_t batch, int32_t n_layers, int32_t n_kv_heads, int32_t layer,
                                  const void *q, int32_t n_q_heads, const int32_t *q_pos,
                                  const int32_t *cache_len, float scale, float *out,
                                  void *workspace, size_t workspace_bytes, int32_t *err_flag,
                                  hipStream_t stream) {
  prcr_status st = check_rope(rope);
  if (st != PRCR_OK) return st;
  if (dtype != PRCR_F32 && dtype != PRCR_BF16) return PRCR_ERR_DTYPE;
  int n_split = 0;
  st = decode_shape(cache, batch, n_q_heads, n_kv_heads, rope->head_dim, &n_split);
  if (st != PRCR_OK) return st;
  st = check_cache(cache);
  if (st != PRCR_OK) return st;
  if (q == nullptr || q_pos == nullptr || cache_len == nullptr || out == nullptr ||
      workspace == nullptr)
    return PRCR_ERR_NULL;
  if (n_layers < 1 || layer < 0 || layer >= n_layers || !std::isfinite(scale)) return PRCR_ERR_SHAPE;
  const size_t need = static_cast<size_t>(batch) * n_q_heads * n_split * (rope->head_dim + 2) * sizeof(float);
  if (workspace_bytes < need) return PRCR_ERR_SHAPE;
  if (!aligned(q, 16) || !aligned(q_pos, 4) || !aligned(cache_len, 4) || !aligned(out, 4) ||
      !aligned(workspace, 4) || (err_flag != nullptr && !aligned(err_flag, 4)))
    return PRCR_ERR_ALIGN;
  DecodeParams p{};
  p.q = q;
  p.q_pos = q_pos;
  p.cache_len = cache_len;
  p.cache_k = cache->k;
  p.cache_v = cache->v;
  p.block_table = cache->block_table;
  p.out = out;
  p.ws = static_cast<float *>(workspace);
  p.err = err_flag;
  p.batch = batch;
  p.n_layers = n_layers;
  p.n_kv_heads = n_kv_heads;
  p.n_q_heads = n_q_heads;
  p.layer = layer;
  p.s_max = cache->s_max;
  p.block_size = cache->block_size;
  p.max_blocks = cache->max_blocks;
  p.n_blocks = cache->n_blocks;
  p.block_shift = -1;
  if (cache->paged && (cache->block_size & (cache->block_size - 1)) == 0)
    for (int sh = 0; sh < 31; ++sh)
      if ((1 << sh) == cache->block_size) p.block_shift = sh;
  p.n_split = n_split;
  p.scale = scale;
  for (int i = 0; i < rope->head_dim / 2; ++i)
    p.inv_freq[i] = std::pow(rope->theta, -(2.0 * i) / rope->head_dim);
  const hipError_t e = launch_decode(p, dtype, rope->head_dim, cache->paged != 0, stream);
  return launch_status(e);
}

prcr_status prcr_revisit(const prcr_rope *rope, const prcr_mem *mem, const int32_t *sel_off,
                         const int32_t *sel_idx, int32_t total_k, const int32_t *p_txt,
                         prcr_mode mode, int32_t l_ext, const prcr_cache *cache,
                         const int32_t *cache_len, double *new_pos, int32_t *next_pos,
                         int32_t *new_cache_len, int64_t *slot_mapping, int32_t *err_flag,
                         hipStream_t stream) {
  RebindParams p;
  AxisMapId map;
  const prcr_status st = prepare_rebind(rope, mem, sel_off, sel_idx, total_k, cache, cache_len,
                                        new_cache_len, slot_mapping, err_flag, true, &p, &map);
  if (st != PRCR_OK) return st;
  if (p_txt == nullptr || next_pos == nullptr) return PRCR_ERR_NULL;
  if (mode < PRCR_MODE_PCR || mode > PRCR_MODE_PCR_RIGHT || l_ext < 0) return PRCR_ERR_MODE;
  if (!aligned(p_txt, 4) || !aligned(next_pos, 4) || (new_pos != nullptr && !aligned(new_pos, 8)))
    return PRCR_ERR_ALIGN;
  p.coords = mem->coords;
  p.p_txt = p_txt;
  p.pos_out = new_pos;
  p.next_pos = next_pos;
  p.mode = static_cast<int32_t>(mode);
  p.l_ext = l_ext;
  const hipError_t e = launch_rebind(p, mem->dtype, mem->head_dim, map, cache->paged != 0, true, stream);
  return launch_status(e);
}

}  // extern "C"
