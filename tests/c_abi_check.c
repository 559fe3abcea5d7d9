/*
 * A plain C consumer of the library: no Python, no torch, only HIP memory calls
 * and the functions include/prcr.h declares.  It runs one small prompt through
 * prefill capture (Eq. (4), (6)-(7)), revisits every visual token at its
 * original coordinates (IDENTITY reassignment, then rebind and inject,
 * Eq. (11)-(13)), and decodes one step of attention over a one-key cache
 * (Eq. (14)); it checks the properties these calls have by definition:
 *   - a token rebound at its original coordinates gets the key the prefill
 *     wrote for it, bit for bit, and its value row unchanged;
 *   - the new lengths and slots follow Eq. (13)'s concatenation;
 *   - attention over a single key returns that key's value row exactly.
 * Exit status 0 on success; a message names the first failed check.
 *
 * Shapes: 2 sequences, 3 layers, 2 KV heads, head_dim 64, float32, sections
 * [8,12,12]; sequence b has 3 text tokens, a 3 x 4 image, 2 text tokens.
 */
#include <stdio.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "prcr.h"

#define B 2
#define NL 3
#define H 2
#define D 64
#define M 12             /* visual tokens per sequence */
#define S 17             /* prompt rows per sequence: 3 + 12 + 2 */
#define SMAX 40

static int fail(const char *what) {
  fprintf(stderr, "c_abi_check: FAILED: %s\n", what);
  return 1;
}

#define HIP_OK(call) do { if ((call) != hipSuccess) return fail(#call); } while (0)
#define PRCR_OK_(call) do { prcr_status st_ = (call); \
    if (st_ != PRCR_OK) { fprintf(stderr, "%s: %s\n", #call, prcr_status_str(st_)); return 1; } } while (0)

static uint32_t lcg = 12345u;
static float next_value(void) {             /* deterministic values in [-1, 1) */
  lcg = lcg * 1664525u + 1013904223u;
  return (float)((lcg >> 8) & 0xFFFF) / 32768.0f - 1.0f;
}

int main(void) {
  /* host inputs: prompt layout and raw projections */
  static int32_t pos[B][S][3], vis[B][S], n_tok[B], n_vis[B], start[B];
  static float raw_k[NL][B][S][H][D], raw_v[NL][B][S][H][D];
  for (int b = 0; b < B; ++b) {
    int s = 0, q = 0;
    for (int i = 0; i < 3; ++i, ++s, ++q) { pos[b][s][0] = pos[b][s][1] = pos[b][s][2] = q; vis[b][s] = -1; }
    for (int h = 0; h < 3; ++h)
      for (int w = 0; w < 4; ++w, ++s) {
        pos[b][s][0] = q; pos[b][s][1] = q + h; pos[b][s][2] = q + w; vis[b][s] = h * 4 + w;
      }
    q += 4;
    for (int i = 0; i < 2; ++i, ++s, ++q) { pos[b][s][0] = pos[b][s][1] = pos[b][s][2] = q; vis[b][s] = -1; }
    n_tok[b] = S; n_vis[b] = M; start[b] = 0;
  }
  for (size_t i = 0; i < sizeof(raw_k) / sizeof(float); ++i) {
    ((float *)raw_k)[i] = next_value();
    ((float *)raw_v)[i] = next_value();
  }

  /* device buffers */
  const size_t mem_bytes = (size_t)B * M * NL * H * D * sizeof(float);
  const size_t cache_bytes = (size_t)B * NL * H * SMAX * D * sizeof(float);
  const size_t raw_bytes = (size_t)B * S * H * D * sizeof(float);
  void *mk, *mv, *ck, *cv, *rk, *rv, *ws;
  int32_t *coords, *nvis, *dpos, *dvis, *dntok, *dstart, *err, *sel_off, *sel_idx, *p_txt, *next_pos,
      *new_len, *qpos, *clen;
  double *new_pos;
  int64_t *slots;
  float *q, *out;
  HIP_OK(hipMalloc(&mk, mem_bytes)); HIP_OK(hipMalloc(&mv, mem_bytes));
  HIP_OK(hipMalloc(&ck, cache_bytes)); HIP_OK(hipMalloc(&cv, cache_bytes));
  HIP_OK(hipMalloc(&rk, raw_bytes)); HIP_OK(hipMalloc(&rv, raw_bytes));
  HIP_OK(hipMalloc((void **)&coords, B * M * 3 * sizeof(int32_t)));
  HIP_OK(hipMalloc((void **)&nvis, sizeof(n_vis)));
  HIP_OK(hipMalloc((void **)&dpos, sizeof(pos))); HIP_OK(hipMalloc((void **)&dvis, sizeof(vis)));
  HIP_OK(hipMalloc((void **)&dntok, sizeof(n_tok))); HIP_OK(hipMalloc((void **)&dstart, sizeof(start)));
  HIP_OK(hipMalloc((void **)&err, sizeof(int32_t)));
  HIP_OK(hipMemset(ck, 0, cache_bytes)); HIP_OK(hipMemset(cv, 0, cache_bytes));
  HIP_OK(hipMemset(err, 0, sizeof(int32_t)));
  HIP_OK(hipMemcpy(nvis, n_vis, sizeof(n_vis), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dpos, pos, sizeof(pos), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dvis, vis, sizeof(vis), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dntok, n_tok, sizeof(n_tok), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(dstart, start, sizeof(start), hipMemcpyHostToDevice));

  prcr_rope rope = {D, {8, 12, 12}, 0, 1e6};
  prcr_mem mem = {mk, mv, coords, nvis, B, M, NL, H, D, PRCR_F32, NULL};
  prcr_cache cache = {0, ck, cv, SMAX, NULL, 0, 0, 0};

  /* prefill capture, one layer at a time */
  for (int l = 0; l < NL; ++l) {
    HIP_OK(hipMemcpy(rk, raw_k[l], raw_bytes, hipMemcpyHostToDevice));
    HIP_OK(hipMemcpy(rv, raw_v[l], raw_bytes, hipMemcpyHostToDevice));
    PRCR_OK_(prcr_prefill_capture(&rope, &mem, l, rk, rv, S, dpos, dntok, dvis, 1, &cache, dstart,
                                  err, NULL));
  }

  /* revisit every visual token of both sequences at its original coordinates */
  int32_t h_off[B + 1], h_idx[B * M], h_ptxt[B];
  for (int b = 0; b <= B; ++b) h_off[b] = b * M;
  for (int i = 0; i < B * M; ++i) h_idx[i] = i % M;
  for (int b = 0; b < B; ++b) h_ptxt[b] = pos[b][S - 1][0];
  HIP_OK(hipMalloc((void **)&sel_off, sizeof(h_off))); HIP_OK(hipMalloc((void **)&sel_idx, sizeof(h_idx)));
  HIP_OK(hipMalloc((void **)&p_txt, sizeof(h_ptxt))); HIP_OK(hipMalloc((void **)&next_pos, B * sizeof(int32_t)));
  HIP_OK(hipMalloc((void **)&new_len, B * sizeof(int32_t)));
  HIP_OK(hipMalloc((void **)&new_pos, B * M * 3 * sizeof(double)));
  HIP_OK(hipMalloc((void **)&slots, B * M * sizeof(int64_t)));
  HIP_OK(hipMemcpy(sel_off, h_off, sizeof(h_off), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(sel_idx, h_idx, sizeof(h_idx), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(p_txt, h_ptxt, sizeof(h_ptxt), hipMemcpyHostToDevice));
  PRCR_OK_(prcr_reassign_coords(&mem, sel_off, sel_idx, B * M, p_txt, PRCR_MODE_IDENTITY, 2, new_pos,
                                next_pos, err, NULL));
  PRCR_OK_(prcr_rebind_inject(&rope, &mem, sel_off, sel_idx, B * M, new_pos, &cache, dntok, new_len,
                              slots, err, NULL));
  HIP_OK(hipDeviceSynchronize());

  int32_t h_err = -1, h_new_len[B], h_next[B];
  int64_t h_slots[B * M];
  HIP_OK(hipMemcpy(&h_err, err, sizeof(int32_t), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_new_len, new_len, sizeof(h_new_len), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_next, next_pos, sizeof(h_next), hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(h_slots, slots, sizeof(h_slots), hipMemcpyDeviceToHost));
  if (h_err != 0) return fail("device data error flag");
  float *hk = malloc(cache_bytes), *hv = malloc(cache_bytes);
  if (!hk || !hv) return fail("host allocation");
  HIP_OK(hipMemcpy(hk, ck, cache_bytes, hipMemcpyDeviceToHost));
  HIP_OK(hipMemcpy(hv, cv, cache_bytes, hipMemcpyDeviceToHost));
  for (int b = 0; b < B; ++b) {
    if (h_new_len[b] != S + M) return fail("new cache length");
    if (h_next[b] != h_ptxt[b] + 1) return fail("next text position");
    for (int s = 0; s < S; ++s) {
      const int m = vis[b][s];
      if (m < 0) continue;
      const int slot = S + m;                       /* token j = m of the selection */
      if (h_slots[b * M + m] != (int64_t)b * SMAX + slot) return fail("slot mapping");
      for (int l = 0; l < NL; ++l)
        for (int h = 0; h < H; ++h) {
          const size_t a = ((((size_t)b * NL + l) * H + h) * SMAX + s) * D;
          const size_t c = ((((size_t)b * NL + l) * H + h) * SMAX + slot) * D;
          if (memcmp(hk + a, hk + c, D * sizeof(float)) != 0) return fail("rebound key differs from prefill key");
          if (memcmp(hv + c, raw_v[l][b][s][h], D * sizeof(float)) != 0) return fail("value row changed");
        }
    }
  }

  /* decode over a one-key cache: the output is that key's value row */
  int32_t h_qpos[B] = {50, 7}, h_clen[B] = {1, 1};
  size_t ws_bytes = 0;
  PRCR_OK_(prcr_decode_workspace_size(&cache, B, 2 * H, H, D, &ws_bytes));
  HIP_OK(hipMalloc(&ws, ws_bytes));
  HIP_OK(hipMalloc((void **)&q, (size_t)B * 2 * H * D * sizeof(float)));
  HIP_OK(hipMalloc((void **)&out, (size_t)B * 2 * H * D * sizeof(float)));
  HIP_OK(hipMalloc((void **)&qpos, sizeof(h_qpos))); HIP_OK(hipMalloc((void **)&clen, sizeof(h_clen)));
  float hq[B * 2 * H * D];
  for (int i = 0; i < B * 2 * H * D; ++i) hq[i] = next_value();
  HIP_OK(hipMemcpy(q, hq, sizeof(hq), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(qpos, h_qpos, sizeof(h_qpos), hipMemcpyHostToDevice));
  HIP_OK(hipMemcpy(clen, h_clen, sizeof(h_clen), hipMemcpyHostToDevice));
  PRCR_OK_(prcr_decode_attention(&rope, &cache, PRCR_F32, B, NL, H, 1, q, 2 * H, qpos, clen, 0.125f, out,
                                 ws, ws_bytes, err, NULL));
  HIP_OK(hipDeviceSynchronize());
  float hout[B * 2 * H * D];
  HIP_OK(hipMemcpy(hout, out, sizeof(hout), hipMemcpyDeviceToHost));
  for (int b = 0; b < B; ++b)
    for (int qh = 0; qh < 2 * H; ++qh) {
      const size_t c = ((((size_t)b * NL + 1) * H + qh / 2) * SMAX + 0) * D;   /* layer 1, slot 0 */
      if (memcmp(hout + ((size_t)b * 2 * H + qh) * D, hv + c, D * sizeof(float)) != 0)
        return fail("one-key attention is not the value row");
    }
  printf("c_abi_check: ok (library version %d)\n", prcr_version());
  return 0;
}
