// extern "C" entry points: structural validation on the host, then one kernel
// launch on the caller's stream.  No entry point allocates or keeps state.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <cstddef>

#include "prcr_internal.h"

using namespace prcr;

namespace {

constexpr int32_t kVersion = 1 * 10000 + 4 * 100 + 0;
constexpr int64_t kMaxDecodeSlots = int64_t{1} << 30;   // decode: cache capacity per sequence

bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Whether the byte ranges [a, a + na) and [b, b + nb) share a byte (null never does).
bool overlaps(const void *a, size_t na, const void *b, size_t nb) {
  if (a == nullptr || b == nullptr || na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

int elem_bytes(prcr_dtype d) { return d == PRCR_F32 ? 4 : 2; }


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

prcr_status prcr::launch_status(hipError_t e) {
  if (e == hipSuccess) return PRCR_OK;
  return e == hipErrorInvalidConfiguration ? PRCR_ERR_SHAPE : PRCR_ERR_HIP;
}

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
    case PRCR_ERR_SCRATCH:
      return "the call needs more scratch memory than the library's static device buffer holds";
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
  // Sequence b's workgroup writes next_pos[b] while the others read their own
  // offsets and visual counts.  (next_pos may alias p_txt: a workgroup reads only
  // its own p_txt[b], before it writes next_pos[b].)
  const size_t nb4 = static_cast<size_t>(mem->batch) * 4;
  if (overlaps(next_pos, nb4, sel_off, nb4 + 4) || overlaps(next_pos, nb4, mem->n_visual, nb4))
    return PRCR_ERR_ALIAS;
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
  // The first workgroup writes the new lengths while the others still read the
  // old lengths and the offsets.
  const size_t nb4 = static_cast<size_t>(mem->batch) * 4;
  if (overlaps(new_cache_len, nb4, cache_len, nb4) || overlaps(new_cache_len, nb4, sel_off, nb4 + 4))
    return PRCR_ERR_ALIAS;
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
  *n_split = decode_splits(cap, batch, n_kv_heads, n_q_heads / n_kv_heads);
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

}  // extern "C"

prcr_status prcr::prepare_decode(const prcr_rope *rope, const prcr_cache *cache, prcr_dtype dtype,
                                 int32_t batch, int32_t n_layers, int32_t n_kv_heads, int32_t layer,
                                 const void *q, int32_t n_q_heads, const int32_t *q_pos,
                                 const int32_t *cache_len, float scale, float *out,
                                 int32_t *err_flag, DecodeParams *out_params, size_t *ws_bytes) {
  prcr_status st = check_rope(rope);
  if (st != PRCR_OK) return st;
  if (dtype != PRCR_F32 && dtype != PRCR_BF16) return PRCR_ERR_DTYPE;
  int n_split = 0;
  st = decode_shape(cache, batch, n_q_heads, n_kv_heads, rope->head_dim, &n_split);
  if (st != PRCR_OK) return st;
  st = check_cache(cache);
  if (st != PRCR_OK) return st;
  if (q == nullptr || q_pos == nullptr || cache_len == nullptr || out == nullptr) return PRCR_ERR_NULL;
  if (n_layers < 1 || layer < 0 || layer >= n_layers || !std::isfinite(scale)) return PRCR_ERR_SHAPE;
  if (!aligned(q, 16) || !aligned(q_pos, 4) || !aligned(cache_len, 4) || !aligned(out, 4) ||
      (err_flag != nullptr && !aligned(err_flag, 4)))
    return PRCR_ERR_ALIGN;
  *ws_bytes = static_cast<size_t>(batch) * n_q_heads * n_split * (rope->head_dim + 2) * sizeof(float);
  DecodeParams &p = *out_params;
  p = DecodeParams{};
  p.q = q;
  p.q_pos = q_pos;
  p.cache_len = cache_len;
  p.cache_k = cache->k;
  p.cache_v = cache->v;
  p.block_table = cache->block_table;
  p.out = out;
  p.ws = nullptr;
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
  return PRCR_OK;
}

extern "C" {

prcr_status prcr_decode_attention(const prcr_rope *rope, const prcr_cache *cache, prcr_dtype dtype,
                                  int32_t batch, int32_t n_layers, int32_t n_kv_heads, int32_t layer,
                                  const void *q, int32_t n_q_heads, const int32_t *q_pos,
                                  const int32_t *cache_len, float scale, float *out,
                                  void *workspace, size_t workspace_bytes, int32_t *err_flag,
                                  hipStream_t stream) {
  DecodeParams p;
  size_t need = 0;
  const prcr_status st = prepare_decode(rope, cache, dtype, batch, n_layers, n_kv_heads, layer, q,
                                        n_q_heads, q_pos, cache_len, scale, out, err_flag, &p, &need);
  if (st != PRCR_OK) return st;
  if (workspace == nullptr) return PRCR_ERR_NULL;
  if (workspace_bytes < need) return PRCR_ERR_SHAPE;
  if (!aligned(workspace, 4)) return PRCR_ERR_ALIGN;
  p.ws = static_cast<float *>(workspace);
  return launch_status(launch_decode(p, dtype, rope->head_dim, cache->paged != 0, stream));
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
  // One wave per sequence writes next_pos[b] (and the first workgroup the new
  // lengths) while every other wave of the launch still reads p_txt, cache_len,
  // the offsets and the visual counts: none of them may share memory with an
  // output, and the two outputs may not share memory with each other.  (An
  // in-place advance of p_txt needs the two-call path or a separate buffer.)
  const size_t nb4 = static_cast<size_t>(mem->batch) * 4;
  if (overlaps(next_pos, nb4, p_txt, nb4) || overlaps(next_pos, nb4, cache_len, nb4) ||
      overlaps(next_pos, nb4, sel_off, nb4 + 4) || overlaps(next_pos, nb4, mem->n_visual, nb4) ||
      overlaps(next_pos, nb4, new_cache_len, nb4) || overlaps(new_cache_len, nb4, p_txt, nb4))
    return PRCR_ERR_ALIAS;
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
