// Host-side checks of the C ABI's argument handling, built with the address and
// undefined-behaviour sanitizers (no GPU, no HIP runtime): api.cpp and
// axis_map.cpp are linked against stub launchers that record what they were
// handed instead of launching.  Every entry point gets malformed arguments
// (null, misaligned, out-of-range and overflow-sized values) and well-formed
// ones; for the latter the recorded launch parameters are checked.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "prcr_internal.h"

namespace prcr {
// --- stub launchers: record the last call -------------------------------------
static int g_calls = 0;
static RebindParams g_rebind;
static ReassignParams g_reassign;
static DecodeParams g_decode;
static PrefillParams g_prefill;
static StoreParams g_store;
static bool g_fused = false;
hipError_t launch_reassign(const ReassignParams &p, hipStream_t) { ++g_calls; g_reassign = p; return hipSuccess; }
hipError_t launch_rebind(const RebindParams &p, prcr_dtype, int, AxisMapId, bool, bool fused, hipStream_t) {
  ++g_calls; g_rebind = p; g_fused = fused; return hipSuccess;
}
hipError_t launch_store(const StoreParams &p, hipStream_t) { ++g_calls; g_store = p; return hipSuccess; }
hipError_t launch_prefill(const PrefillParams &p, prcr_dtype, int, AxisMapId, bool, hipStream_t) {
  ++g_calls; g_prefill = p; return hipSuccess;
}
hipError_t launch_decode(const DecodeParams &p, prcr_dtype, int, bool, hipStream_t) {
  ++g_calls; g_decode = p; return hipErrorInvalidValue;     // a launch failure maps to PRCR_ERR_HIP
}
int decode_splits(int64_t, int, int, int) { return 3; }
}  // namespace prcr

using namespace prcr;

static int failures = 0;
#define EXPECT(cond) do { if (!(cond)) { std::fprintf(stderr, "FAILED line %d: %s\n", __LINE__, #cond); ++failures; } } while (0)

// 256-byte aligned placeholder addresses inside one host buffer: never dereferenced
// by the library, which only validates and forwards them.
alignas(256) static unsigned char arena[1 << 16];
static void *at(size_t off) { return arena + off; }

int main() {
  prcr_rope rope = {128, {16, 24, 24}, 0, 1e6};
  prcr_mem mem = {at(0), at(256), reinterpret_cast<int32_t *>(at(512)), reinterpret_cast<int32_t *>(at(768)),
                  2, 100, 28, 4, 128, PRCR_BF16, nullptr};
  prcr_cache cache = {0, at(1024), at(1280), 512, nullptr, 0, 0, 0};
  const int32_t *off = reinterpret_cast<int32_t *>(at(2048));
  const int32_t *idx = reinterpret_cast<int32_t *>(at(2304));
  const int32_t *ptxt = reinterpret_cast<int32_t *>(at(2560));
  const int32_t *clen = reinterpret_cast<int32_t *>(at(2816));
  int32_t *nlen = reinterpret_cast<int32_t *>(at(3072));
  int32_t *nextp = reinterpret_cast<int32_t *>(at(3328));
  double *npos = reinterpret_cast<double *>(at(3584));
  int64_t *slots = reinterpret_cast<int64_t *>(at(3840));
  int32_t *err = reinterpret_cast<int32_t *>(at(4096));

  // --- status strings and host tables ------------------------------------------
  for (int s = 0; s <= 9; ++s) EXPECT(prcr_status_str(static_cast<prcr_status>(s)) != nullptr);
  double invf[64];
  EXPECT(prcr_inv_freq(&rope, invf) == PRCR_OK);
  for (int i = 0; i < 64; ++i) EXPECT(invf[i] == std::pow(1e6, -(2.0 * i) / 128));
  int32_t axis[64];
  EXPECT(prcr_pair_axis(&rope, axis) == PRCR_OK);
  EXPECT(axis[0] == 0 && axis[15] == 0 && axis[16] == 1 && axis[39] == 1 && axis[40] == 2 && axis[63] == 2);
  prcr_rope odd = {128, {32, 16, 16}, 0, 1e6};
  EXPECT(prcr_pair_axis(&odd, axis) == PRCR_ERR_UNSUPPORTED);
  prcr_rope inf_theta = {128, {16, 24, 24}, 0, INFINITY};
  EXPECT(prcr_inv_freq(&inf_theta, invf) == PRCR_ERR_SHAPE);

  // --- rebind: malformed --------------------------------------------------------
  auto rebind = [&](const prcr_rope *r, const prcr_mem *m, int total_k, const prcr_cache *c,
                    int32_t *nl = nullptr) {
    return prcr_rebind_inject(r, m, off, idx, total_k, npos, c, clen, nl ? nl : nlen, slots, err, nullptr);
  };
  EXPECT(rebind(nullptr, &mem, 10, &cache) == PRCR_ERR_NULL);
  EXPECT(rebind(&rope, nullptr, 10, &cache) == PRCR_ERR_NULL);
  EXPECT(rebind(&rope, &mem, 10, nullptr) == PRCR_ERR_NULL);
  EXPECT(rebind(&rope, &mem, -1, &cache) == PRCR_ERR_SHAPE);
  EXPECT(rebind(&rope, &mem, 10, &cache, const_cast<int32_t *>(clen)) == PRCR_ERR_ALIAS);
  {
    prcr_mem m = mem; m.n_layers = INT32_MAX; m.n_kv_heads = INT32_MAX;   // overflow-sized rows
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_SHAPE);
    m = mem; m.head_dim = INT32_MAX;
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_SHAPE);
    m = mem; m.batch = INT32_MIN;
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_SHAPE);
    m = mem; m.dtype = static_cast<prcr_dtype>(-7);
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_DTYPE);
    m = mem; m.k = at(8);
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_ALIGN);
    m = mem; m.v = nullptr;                                                // key-only without a slot table
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_NULL);
    m.v_slot = reinterpret_cast<int32_t *>(at(4354));                      // misaligned slot table
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_ERR_ALIGN);
    prcr_cache c = cache; c.s_max = INT32_MIN;
    EXPECT(rebind(&rope, &mem, 10, &c) == PRCR_ERR_SHAPE);
    c = cache; c.paged = 1; c.block_table = reinterpret_cast<int32_t *>(at(4608));
    c.block_size = INT32_MAX; c.max_blocks = INT32_MAX; c.n_blocks = 1;
    EXPECT(rebind(&rope, &mem, 10, &c) == PRCR_OK);                        // geometry is device-checked
    prcr_rope r = rope; r.section[0] = INT32_MAX;
    EXPECT(rebind(&r, &mem, 10, &cache) == PRCR_ERR_SHAPE);
    r = rope; r.head_dim = -128;
    EXPECT(rebind(&r, &mem, 10, &cache) == PRCR_ERR_SHAPE);
  }

  // --- rebind and revisit: well formed -------------------------------------------
  g_calls = 0;
  EXPECT(rebind(&rope, &mem, 10, &cache) == PRCR_OK);
  EXPECT(g_calls == 1 && !g_fused);
  EXPECT(g_rebind.total_k == 10 && g_rebind.batch == 2 && g_rebind.n_layers == 28 && g_rebind.n_kv_heads == 4);
  EXPECT(g_rebind.s_max == 512 && g_rebind.new_pos == npos && g_rebind.v_slot == nullptr);
  for (int i = 0; i < 64; ++i) EXPECT(g_rebind.inv_freq[i] == std::pow(1e6, -(2.0 * i) / 128));
  {
    prcr_mem m = mem; m.v = nullptr; m.v_slot = reinterpret_cast<int32_t *>(at(4352));
    EXPECT(rebind(&rope, &m, 10, &cache) == PRCR_OK);
    EXPECT(g_rebind.mem_v == nullptr && g_rebind.v_slot == m.v_slot);
  }
  EXPECT(prcr_revisit(&rope, &mem, off, idx, 10, ptxt, PRCR_MODE_SHIFT, 2, &cache, clen, npos, nextp, nlen,
                      slots, err, nullptr) == PRCR_OK);
  EXPECT(g_fused && g_rebind.mode == PRCR_MODE_SHIFT && g_rebind.l_ext == 2 && g_rebind.next_pos == nextp);
  EXPECT(prcr_revisit(&rope, &mem, off, idx, 10, ptxt, static_cast<prcr_mode>(99), 2, &cache, clen, npos,
                      nextp, nlen, slots, err, nullptr) == PRCR_ERR_MODE);

  // --- reassign --------------------------------------------------------------------
  EXPECT(prcr_reassign_coords(&mem, off, idx, 10, ptxt, PRCR_MODE_PCR, 2, npos, nextp, err, nullptr) == PRCR_OK);
  EXPECT(g_reassign.total_k == 10 && g_reassign.mode == PRCR_MODE_PCR && g_reassign.l_ext == 2);
  EXPECT(prcr_reassign_coords(&mem, off, idx, 10, ptxt, PRCR_MODE_PCR, -1, npos, nextp, err, nullptr) ==
         PRCR_ERR_MODE);
  EXPECT(prcr_reassign_coords(&mem, off, idx, 10, ptxt, PRCR_MODE_PCR, 2, nullptr, nextp, err, nullptr) ==
         PRCR_ERR_NULL);
  EXPECT(prcr_reassign_coords(&mem, off, idx, 0, ptxt, PRCR_MODE_PCR, 2, nullptr, nextp, err, nullptr) ==
         PRCR_OK);                                                         // nothing selected: no positions

  // --- store and prefill -------------------------------------------------------------
  EXPECT(prcr_store_raw(&mem, 27, at(5120), at(5376), 40, idx, err, nullptr) == PRCR_OK);
  EXPECT(g_store.layer == 27 && g_store.row_bytes == 4 * 128 * 2);
  EXPECT(prcr_store_raw(&mem, 28, at(5120), at(5376), 40, idx, err, nullptr) == PRCR_ERR_SHAPE);
  {
    prcr_mem m = mem; m.n_layers = 1; m.n_kv_heads = 1 << 24;   // a token row of 2^32 bytes
    EXPECT(prcr_store_raw(&m, 0, at(5120), at(5376), 40, idx, err, nullptr) == PRCR_ERR_SHAPE);
  }
  {
    prcr_mem m = mem; m.v = nullptr; m.v_slot = reinterpret_cast<int32_t *>(at(4352));
    EXPECT(prcr_store_raw(&m, 0, at(5120), nullptr, 40, idx, err, nullptr) == PRCR_OK);   // keys only
    EXPECT(g_store.raw_v == nullptr && g_store.mem_v == nullptr);
    EXPECT(prcr_prefill_capture(&rope, &m, 3, at(5120), at(5376), 40, ptxt, clen, idx, 1, &cache, clen, err,
                                nullptr) == PRCR_OK);
    EXPECT(g_prefill.v_slot == m.v_slot && g_prefill.layer == 3 && g_prefill.write_coords == 1);
  }
  EXPECT(prcr_prefill_capture(&rope, &mem, 3, at(5120), at(5376), 0, ptxt, clen, idx, 1, &cache, clen, err,
                              nullptr) == PRCR_ERR_SHAPE);

  // --- decode -----------------------------------------------------------------------
  size_t ws = 0;
  EXPECT(prcr_decode_workspace_size(&cache, 2, 16, 4, 128, &ws) == PRCR_OK);
  EXPECT(ws == static_cast<size_t>(2) * 16 * 3 * (128 + 2) * sizeof(float));    // 3 splits from the stub
  EXPECT(prcr_decode_workspace_size(&cache, 65536, 16, 4, 128, &ws) == PRCR_ERR_SHAPE);
  EXPECT(prcr_decode_workspace_size(&cache, 2, INT32_MAX, 1, 128, &ws) == PRCR_ERR_SHAPE);
  float *out = reinterpret_cast<float *>(at(6144));
  const void *q = at(6400);
  EXPECT(prcr_decode_attention(&rope, &cache, PRCR_BF16, 2, 28, 4, 5, q, 16, ptxt, clen, 0.088f, out, at(8192),
                               ws, err, nullptr) == PRCR_ERR_HIP);         // the stub's launch failure
  EXPECT(g_decode.n_split == 3 && g_decode.layer == 5 && g_decode.n_q_heads == 16 && g_decode.scale == 0.088f);
  EXPECT(prcr_decode_attention(&rope, &cache, PRCR_BF16, 2, 28, 4, 5, q, 16, ptxt, clen, 0.088f, out, at(8192),
                               ws - 4, err, nullptr) == PRCR_ERR_SHAPE);   // workspace one float short
  EXPECT(prcr_decode_attention(&rope, &cache, PRCR_BF16, 2, 28, 4, 5, q, 16, ptxt, clen, NAN, out, at(8192),
                               ws, err, nullptr) == PRCR_ERR_SHAPE);

  if (failures == 0) std::printf("host_abi_check: ok\n");
  return failures == 0 ? 0 : 1;
}
