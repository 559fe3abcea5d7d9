/*
 * prcr.h - C ABI of the MI355X (gfx950) position-rebinding cache-reuse library.
 *
 * Position Rebinding Cache Reuse (PRCR) revisits visual evidence during decoding
 * without replaying visual tokens through the model (Sec. 3, Algorithm 1):
 *
 *   1. the raw (pre-rotary) K/V projections of every visual token are kept for
 *      every layer together with the token's original coordinates - the Raw
 *      Visual Evidence Memory, Eq. (6)-(7);                  -> prcr_store_raw
 *   2. the selected tokens get new coordinates next to the current text
 *      position - Position-Consistent Reinsertion, Eq. (8)-(10); -> prcr_reassign_coords
 *   3. their raw keys are rotated at the new coordinates, values are reused
 *      unchanged (Eq. (11)-(12)), and both are appended to the active decoder
 *      cache (Eq. (13)).                                     -> prcr_rebind_inject
 *
 * Conventions shared by every entry point
 *   - Every pointer inside the structs and every array argument is a DEVICE
 *     pointer unless marked "host".  The structs themselves are host memory and
 *     are read only during the call.
 *   - Calls are asynchronous on `stream`.  The caller owns all buffers and keeps
 *     them alive until the stream work completes.  The library keeps no state
 *     between calls and allocates no memory; calls are re-entrant.  (The one
 *     exception is the static device scratch array of
 *     prcr_decode_attention_static, see there.)
 *   - Structural errors (null pointer, bad shape, misalignment, unsupported
 *     combination) are detected on the host before any HIP call and returned;
 *     nothing is launched and no output is touched.  A problem too large for
 *     one launch (a grid dimension beyond 2^32 - 1 work-items, which the dispatch
 *     cannot express) is such an error too: PRCR_ERR_SHAPE.  A failed kernel
 *     launch returns PRCR_ERR_HIP.
 *   - Data errors found on the device (an index outside the visual-token range,
 *     a slot beyond the cache capacity, a block-table entry outside the pool,
 *     malformed selection offsets, a position outside the exact range) OR their
 *     PRCR_DERR_* bit into *err_flag when err_flag is non-NULL.  The affected row
 *     is skipped: no access ever goes out of the bounds the arguments describe.
 *     Clear *err_flag before the call if a fresh report is wanted.
 *   - Element types: K, V of the memory, the raw projections and the cache share
 *     `dtype` (float32 or bfloat16).  Every K/V base pointer is 16-byte aligned,
 *     int32 arrays 4-byte, int64 and double arrays 8-byte aligned.
 *
 * Layouts (row-major, innermost last)
 *   memory K / V       [batch][max_visual][n_layers][n_kv_heads][head_dim]
 *                      (per visual token, its per-layer K/V rows: Eq. (7)'s
 *                      "token -> {(k, v) per layer}, coordinate" record)
 *   memory coords      int32 [batch][max_visual][3]   original (t, h, w)
 *   selection          CSR: sel_off int32 [batch+1] (sel_off[0] = 0,
 *                      non-decreasing, sel_off[batch] = total_k), sel_idx int32
 *                      [total_k]; the order inside a sequence is the injection
 *                      order (slot cache_len[b] + j for its j-th token)
 *   new positions      double [total_k][3]   (t, h, w)
 *   contiguous cache   [batch][n_layers][n_kv_heads][s_max][head_dim]
 *   paged cache        [n_layers][n_blocks][block_size][n_kv_heads][head_dim]
 *                      with block_table int32 [batch][max_blocks]
 *   slot_mapping       int64 [total_k]: contiguous b*s_max + slot,
 *                      paged block*block_size + offset, -1 for a skipped row
 */
#ifndef PRCR_H
#define PRCR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enumerations below are 32-bit integers on both sides of the ABI.  Compiled
 * as C++ they are given int32_t as their underlying type, so that any 32-bit
 * value a C caller passes is a representable value the library can reject
 * (rather than an out-of-range enumeration value). */
#ifdef __cplusplus
#define PRCR_ENUM_BASE : int32_t
#else
#define PRCR_ENUM_BASE
#endif

typedef enum prcr_status PRCR_ENUM_BASE {
  PRCR_OK = 0,
  PRCR_ERR_NULL = 1,          /* a required pointer is NULL                        */
  PRCR_ERR_SHAPE = 2,         /* a size or count is out of range or inconsistent   */
  PRCR_ERR_DTYPE = 3,         /* unknown element type                              */
  PRCR_ERR_ALIGN = 4,         /* a pointer is not aligned as required              */
  PRCR_ERR_MODE = 5,          /* unknown reassignment mode or negative l_ext       */
  PRCR_ERR_UNSUPPORTED = 6,   /* no compiled kernel for this head_dim/axis map     */
  PRCR_ERR_ALIAS = 7,         /* an output aliases an input it must not alias      */
  PRCR_ERR_HIP = 8,           /* the HIP runtime reported a launch error           */
  PRCR_ERR_SCRATCH = 9        /* the call needs more than the library's static
                                 scratch buffer (prcr_decode_attention_static)     */
} prcr_status;

typedef enum prcr_dtype PRCR_ENUM_BASE { PRCR_F32 = 0, PRCR_BF16 = 1 } prcr_dtype;

/* Reassignment rules (Sec. 3.2, Table 2). */
typedef enum prcr_mode PRCR_ENUM_BASE {
  PRCR_MODE_PCR = 0,       /* Position-Consistent Reinsertion, Eq. (8)-(10) (default)    */
  PRCR_MODE_SHIFT = 1,     /* region translated to start at p_txt + 1, layout kept       */
  PRCR_MODE_IDENTITY = 2,  /* original coordinates (direct reuse, Eq. (4))               */
  PRCR_MODE_LPA = 3,       /* Linear Position Appending: p_txt + j                       */
  PRCR_MODE_UIR = 4,       /* Uniform Interval Reinsertion: p_txt + j / (K + 1)          */
  PRCR_MODE_PCR_RIGHT = 5  /* PCR re-anchored rightward (the direction ablation, Sec. 4):
                              Eq. (10) with p_txt + 1 in place of p_txt - L, so entries lie
                              in (p_txt + 1, p_txt + L + 2); next text position p_txt + 1 */
} prcr_mode;

/* Device-side data error bits (OR-ed into *err_flag). */
#define PRCR_DERR_INDEX    1   /* selected index / source row outside its range          */
#define PRCR_DERR_CAPACITY 2   /* slot beyond s_max or beyond max_blocks * block_size     */
#define PRCR_DERR_BLOCK    4   /* block-table entry outside [0, n_blocks)                */
#define PRCR_DERR_OFFSETS  8   /* sel_off not a valid CSR offset array for total_k       */
#define PRCR_DERR_RANGE   16   /* a PCR/UIR position outside the exactly-rounded range   */

/* Multimodal rotary embedding (M-RoPE).  Rotary pair i = (x_i, x_{i+head_dim/2})
 * turns by angle p_axis(i) * theta^(-2i/head_dim).  axis(i): with
 * interleaved = 0, t for i < section[0], h for i < section[0]+section[1], w
 * otherwise; with interleaved = 1, h if i % 3 == 1 and i < 3*section[1], w if
 * i % 3 == 2 and i < 3*section[2], t otherwise.  section[] sums to head_dim/2. */
typedef struct prcr_rope {
  int32_t head_dim;
  int32_t section[3];
  int32_t interleaved;
  double theta;
} prcr_rope;

/* Raw Visual Evidence Memory, Eq. (7).
 *
 * Key-only memory: Eq. (7) keeps both raw rows, but a value row is not rotated
 * (Eq. (4)), so the value the prefill wrote into the standard cache is already
 * the raw value.  With v == NULL the memory keeps keys only (half the bytes)
 * and v_slot[b][m] names the slot of sequence b's standard cache (counted as
 * cache_len counts slots, contiguous or paged) that holds visual token m's
 * value rows for every layer; prcr_prefill_capture fills it.  Revisits then
 * copy the values from that slot of the same cache, which must still hold them
 * and must lie below cache_len[b] (else PRCR_DERR_INDEX and the token is
 * skipped).  With v != NULL, v_slot is ignored and may be NULL. */
typedef struct prcr_mem {
  void *k;                     /* [batch][max_visual][n_layers][n_kv_heads][head_dim] */
  void *v;                     /* same layout, or NULL for a key-only memory          */
  int32_t *coords;             /* int32 [batch][max_visual][3]                          */
  const int32_t *n_visual;     /* int32 [batch], visual tokens stored per sequence     */
  int32_t batch, max_visual, n_layers, n_kv_heads, head_dim;
  prcr_dtype dtype;
  int32_t *v_slot;             /* key-only memory: int32 [batch][max_visual]            */
} prcr_mem;

/* Active decoder cache, Eq. (13).  n_layers, n_kv_heads, head_dim and dtype are
 * those of the memory. */
typedef struct prcr_cache {
  int32_t paged;               /* 0: contiguous, 1: paged                              */
  void *k;                     /* contiguous [batch][n_layers][n_kv_heads][s_max][d]   */
  void *v;                     /* paged [n_layers][n_blocks][block_size][n_kv_heads][d] */
  int32_t s_max;               /* contiguous: slots per sequence                       */
  const int32_t *block_table;  /* paged: int32 [batch][max_blocks]                     */
  int32_t block_size, max_blocks, n_blocks;
} prcr_cache;

/*
 * prcr_store_raw - capture one layer's pre-rotary K/V of the visual tokens
 * into the memory (Sec. 3.1, Eq. (6)-(7)).
 *
 *   raw_k, raw_v  [batch][s_src][n_kv_heads][head_dim]: the layer's K/V
 *                 projections before rotary, as the attention module makes them
 *   vis_rows      int32 [batch][max_visual]: source row of visual token m; only
 *                 m < n_visual[b] are read
 *   layer         0 <= layer < n_layers
 * Writes mem->k/v[b][m][layer] for m < n_visual[b].  A source row outside
 * [0, s_src) is skipped with PRCR_DERR_INDEX.  mem->coords is filled by the
 * caller (it does not depend on the layer).
 */
/* A key-only memory (mem->v == NULL) stores keys only; raw_v may then be NULL
 * and v_slot is the caller's to fill. */
prcr_status prcr_store_raw(const prcr_mem *mem, int32_t layer,
                           const void *raw_k, const void *raw_v, int32_t s_src,
                           const int32_t *vis_rows, int32_t *err_flag,
                           hipStream_t stream);

/*
 * prcr_reassign_coords - new (t, h, w) coordinates for the selected tokens and
 * the next text position (Sec. 3.2, Eq. (8)-(10), Algorithm 1).
 *
 *   sel_off, sel_idx, total_k   CSR selection (see layouts); K_b =
 *                               sel_off[b+1] - sel_off[b] may be 0
 *   p_txt    int32 [batch]: position of the latest text token of sequence b
 *   mode     PRCR_MODE_*; l_ext = the left extension L >= 0 (the paper uses 2)
 *   new_pos  out double [total_k][3]
 *   next_pos out int32 [batch]: position of the next text token
 *
 * PCR, per axis a over the sequence's valid selected tokens: with range
 * [lo, hi], u = (c - lo) / (hi - lo) (u = 1/2 when hi == lo) and
 * p = (p_txt - L) + (L + 1)(1 + (K - 1) u)/(K + 1), the exact rational rounded
 * once to double; next_pos = p_txt + 1.  SHIFT: p = p_txt + 1 + (c - lo),
 * next_pos = max p + 1.  IDENTITY: p = c.  LPA: p = p_txt + j (j = 1..K),
 * next_pos = p_txt + K + 1.  UIR: p = p_txt + j/(K + 1).  A token whose index is
 * outside [0, n_visual[b]) gets NaN positions and PRCR_DERR_INDEX and is left out
 * of the range.  PCR/UIR positions are exact (correctly rounded) while the
 * rational's numerator and denominator stay below 2^52; beyond that the value
 * is within a few ulp and PRCR_DERR_RANGE is raised.  A next text position
 * outside the int32 range is saturated to INT32_MAX (or INT32_MIN), never
 * wrapped, and PRCR_DERR_RANGE is raised.
 *
 * next_pos may be p_txt itself (an in-place advance: each sequence reads its own
 * p_txt before writing its next_pos); it must not share memory with sel_off or
 * n_visual (PRCR_ERR_ALIAS).
 */
prcr_status prcr_reassign_coords(const prcr_mem *mem,
                                 const int32_t *sel_off, const int32_t *sel_idx,
                                 int32_t total_k, const int32_t *p_txt,
                                 prcr_mode mode, int32_t l_ext,
                                 double *new_pos, int32_t *next_pos,
                                 int32_t *err_flag, hipStream_t stream);

/*
 * prcr_rebind_inject - gather the selected memory rows for every layer and KV
 * head (Eq. (11)), rotate the keys at new_pos and reuse the values (Eq. (12)),
 * and append both to the active cache (Eq. (13)), all in one pass.
 *
 *   rope          M-RoPE definition; rope->head_dim == mem->head_dim
 *   new_pos       double [total_k][3] (e.g. from prcr_reassign_coords)
 *   cache_len     int32 [batch] in: first free slot of each sequence
 *   new_cache_len int32 [batch] out (may be NULL): cache_len[b] + K_b; must
 *                 not share memory with cache_len or sel_off (PRCR_ERR_ALIAS)
 *   slot_mapping  int64 [total_k] out (may be NULL)
 *
 * Token j of sequence b goes to slot cache_len[b] + j.  Key elements are
 * rotated in double precision (cos/sin of the double angle) and rounded once to
 * the storage type (round to nearest even); values are copied bit for bit.
 * Compiled axis maps: head_dim 64 with sections [8,12,12] or interleaved
 * [11,11,10]; head_dim 128 with [16,24,24], interleaved [22,21,21] or
 * interleaved [24,20,20]; and 1-D rotary (every pair on t: sections
 * [head_dim/2, 0, 0], either reading) for models with a plain rotary embedding,
 * whose visual tokens carry their 1-D position as t; float32 and bfloat16;
 * contiguous and paged.  With a
 * key-only memory the value rows come from cache slot v_slot[b][m] of the same
 * sequence (see prcr_mem).
 */
prcr_status prcr_rebind_inject(const prcr_rope *rope, const prcr_mem *mem,
                               const int32_t *sel_off, const int32_t *sel_idx,
                               int32_t total_k, const double *new_pos,
                               const prcr_cache *cache, const int32_t *cache_len,
                               int32_t *new_cache_len, int64_t *slot_mapping,
                               int32_t *err_flag, hipStream_t stream);

/*
 * prcr_prefill_capture - one layer of the prompt prefill, fused: reads each
 * prompt token's pre-rotary K/V rows once, writes the rotated key and the value
 * into the standard decoder cache at the token's position ids (Eq. (4)), and
 * writes the raw rows of visual tokens into the memory (Sec. 3.1, Eq. (6)-(7)).
 *
 *   raw_k, raw_v  [batch][s_src][n_kv_heads][head_dim], this layer's projections
 *   pos           int32 [batch][s_src][3]: (t, h, w) position ids of each row
 *   n_tokens      int32 [batch]: rows s < n_tokens[b] are prompt tokens
 *   vis_index     int32 [batch][s_src]: visual token index m of row s, -1 if the
 *                 row is not visual
 *   write_coords  nonzero: also set mem->coords[b][m] = pos[b][s] (their
 *                 original coordinates, used by IDENTITY and as p_m by PCR)
 *   cache_start   int32 [batch]: row s goes to cache slot cache_start[b] + s
 *                 of layer `layer`
 * Keys are rotated as in prcr_rebind_inject (double precision, one rounding),
 * so rebinding a visual token at its original coordinates reproduces the key
 * written here bit for bit.  A slot beyond capacity or a bad block skips the
 * cache row (PRCR_DERR_CAPACITY / _BLOCK); m outside [0, n_visual[b]) or
 * n_tokens[b] outside [0, s_src] raise PRCR_DERR_INDEX.  A key-only memory
 * (mem->v == NULL) gets the raw keys and v_slot[b][m] = cache_start[b] + s.
 */
prcr_status prcr_prefill_capture(const prcr_rope *rope, const prcr_mem *mem, int32_t layer,
                                 const void *raw_k, const void *raw_v, int32_t s_src,
                                 const int32_t *pos, const int32_t *n_tokens,
                                 const int32_t *vis_index, int32_t write_coords,
                                 const prcr_cache *cache, const int32_t *cache_start,
                                 int32_t *err_flag, hipStream_t stream);

/*
 * prcr_revisit - the whole revisit in one launch: reassignment (Eq. (8)-(10),
 * as prcr_reassign_coords) fused with gather, rebinding and injection
 * (Eq. (11)-(13), as prcr_rebind_inject), for callers that revisit a small
 * selection and are bound by launch latency rather than bandwidth (the paper's
 * efficiency study uses K = 32 and 128, Table 3).
 *
 * Arguments are those of the two calls it replaces; new_pos is an optional
 * output here (NULL: positions are not stored).  Results are identical to
 * prcr_reassign_coords followed by prcr_rebind_inject.  Each wavefront reduces
 * its own sequence's coordinate ranges, reading K_b coordinates, so for large
 * selections (hundreds of tokens per sequence and more) the two-call path is
 * faster.
 *
 * Aliasing.  In the single launch, one wave per sequence writes next_pos[b] (and
 * the first workgroup the new lengths) while every other wave still reads p_txt,
 * cache_len, sel_off and n_visual.  So next_pos must not share memory with
 * p_txt, cache_len, sel_off, n_visual or new_cache_len, and new_cache_len not
 * with p_txt, cache_len or sel_off: such calls return PRCR_ERR_ALIAS before any
 * launch.  (Advancing p_txt in place, as a decode loop may, needs a separate
 * next_pos buffer here, or the two-call path.)
 */
prcr_status prcr_revisit(const prcr_rope *rope, const prcr_mem *mem,
                         const int32_t *sel_off, const int32_t *sel_idx, int32_t total_k,
                         const int32_t *p_txt, prcr_mode mode, int32_t l_ext,
                         const prcr_cache *cache, const int32_t *cache_len,
                         double *new_pos, int32_t *next_pos,
                         int32_t *new_cache_len, int64_t *slot_mapping,
                         int32_t *err_flag, hipStream_t stream);

/*
 * prcr_decode_attention - one decode step of attention over the active cache of
 * one layer (Eq. (14)): for each sequence b and query head qh,
 *   out[b][qh] = softmax(scale * RoPE(q[b][qh], (p, p, p)) . K^T) V,
 * p = q_pos[b], over the keys in slots 0 .. cache_len[b]-1 of KV head
 * qh / (n_q_heads / n_kv_heads) (grouped-query attention, at most 8 query heads
 * per KV head).  The next text position of Sec. 3.3 is such a (p, p, p).
 *
 *   cache         contiguous or paged, head_dim = rope->head_dim (64 or 128),
 *                 element type dtype, n_layers / n_kv_heads / batch as given
 *   q             [batch][n_q_heads][head_dim] raw (pre-rotary) queries, dtype
 *   out           float32 [batch][n_q_heads][head_dim]
 *   workspace     at least prcr_decode_workspace_size() bytes of device memory,
 *                 owned by the caller (split-K partial results; no state is kept)
 *   scale         usually 1/sqrt(head_dim)
 * Scores and the softmax are accumulated in float32; the query is rotated in
 * double and rounded to float32 once.  cache_len[b] = 0 gives out = 0.  A
 * cache_len beyond the capacity is clamped with PRCR_DERR_CAPACITY; a block-table
 * entry outside the pool skips its keys with PRCR_DERR_BLOCK.  The capacity per
 * sequence (s_max, or max_blocks * block_size) is at most 2^30 slots, else
 * PRCR_ERR_SHAPE.
 */
prcr_status prcr_decode_attention(const prcr_rope *rope, const prcr_cache *cache,
                                  prcr_dtype dtype, int32_t batch, int32_t n_layers,
                                  int32_t n_kv_heads, int32_t layer,
                                  const void *q, int32_t n_q_heads, const int32_t *q_pos,
                                  const int32_t *cache_len, float scale, float *out,
                                  void *workspace, size_t workspace_bytes,
                                  int32_t *err_flag, hipStream_t stream);

/* Workspace bytes prcr_decode_attention needs for this cache and shape (host). */
prcr_status prcr_decode_workspace_size(const prcr_cache *cache, int32_t batch,
                                       int32_t n_q_heads, int32_t n_kv_heads,
                                       int32_t head_dim, size_t *bytes);

/* Size of the library's static device scratch buffer, per GPU. */
#define PRCR_STATIC_SCRATCH_BYTES ((size_t)16 << 20)

/*
 * prcr_decode_attention_static - prcr_decode_attention without a caller-provided
 * workspace, for callers that cannot allocate device memory at all (code under
 * HIP graph capture, serving loops and harnesses that forbid hipMalloc).  It
 * computes exactly what prcr_decode_attention computes, with the same kernels,
 * the split-K partials going to a static device array that the library holds
 * on every GPU it runs on (PRCR_STATIC_SCRATCH_BYTES each, from the time the
 * library's code is loaded on that GPU until the process ends).  The call
 * allocates nothing, on the host or the device.
 *
 * Arguments and errors are those of prcr_decode_attention; a shape whose
 * partials need more than PRCR_STATIC_SCRATCH_BYTES (prcr_decode_workspace_size
 * tells how much) returns PRCR_ERR_SCRATCH before any HIP call.  The buffer's
 * address on the stream's GPU is looked up on the first call there (a HIP
 * runtime failure then returns PRCR_ERR_HIP).  Every call on one GPU uses the
 * same buffer: calls whose stream work overlaps on one GPU (different streams,
 * or host threads racing on one stream) race on it and give undefined results;
 * calls ordered on one stream, or separated by synchronisation, are safe.  No
 * content is carried from one call to the next (every partial a call reads, it
 * has written).
 */
prcr_status prcr_decode_attention_static(const prcr_rope *rope, const prcr_cache *cache,
                                         prcr_dtype dtype, int32_t batch, int32_t n_layers,
                                         int32_t n_kv_heads, int32_t layer,
                                         const void *q, int32_t n_q_heads,
                                         const int32_t *q_pos, const int32_t *cache_len,
                                         float scale, float *out, int32_t *err_flag,
                                         hipStream_t stream);

/* Host helpers (no GPU work). */

/* Static description of a status code (host). */
const char *prcr_status_str(prcr_status s);

/* The double-precision frequencies theta^(-2i/head_dim), i < head_dim/2, that the
 * kernels use (host; out_host holds head_dim/2 doubles). */
prcr_status prcr_inv_freq(const prcr_rope *rope, double *out_host);

/* The axis (0 = t, 1 = h, 2 = w) of each rotary pair, as the compiled kernels
 * resolve it (host; out_host holds head_dim/2 int32). */
prcr_status prcr_pair_axis(const prcr_rope *rope, int32_t *out_host);

/* Library version as major*10000 + minor*100 + patch (host). */
int32_t prcr_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PRCR_H */
