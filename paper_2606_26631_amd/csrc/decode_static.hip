// prcr_decode_attention_static: decode attention whose split-K partials live in
// a static device array held by the library, for callers that cannot allocate.
//
// The array below is file-scope device memory: every GPU the library's code is
// loaded on holds its own copy at its own address.  Its name, used in host code,
// is only a host-side stand-in for the symbol; host code asks the runtime for the
// device address once per GPU (hipGetSymbolAddress, with that GPU current) and
// passes that address to the kernels, never the name.
#include <mutex>

#include "prcr_internal.h"

namespace {

constexpr size_t kScratchBytes = PRCR_STATIC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

std::mutex g_lock;
void *g_scratch_ptr[kMaxDevices] = {};

// Device address of this GPU's scratch array, looked up on the first call made
// for that GPU (with the GPU made current for the lookup, then restored).
prcr_status scratch_for(int dev, float **out) {
  if (dev < 0 || dev >= kMaxDevices) return PRCR_ERR_HIP;
  std::lock_guard<std::mutex> guard(g_lock);
  if (g_scratch_ptr[dev] == nullptr) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return PRCR_ERR_HIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return PRCR_ERR_HIP;
    void *ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev && hipSetDevice(cur) != hipSuccess) return PRCR_ERR_HIP;
    if (e != hipSuccess || ptr == nullptr) return PRCR_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = static_cast<float *>(g_scratch_ptr[dev]);
  return PRCR_OK;
}

}  // namespace

extern "C" prcr_status prcr_decode_attention_static(
    const prcr_rope *rope, const prcr_cache *cache, prcr_dtype dtype, int32_t batch,
    int32_t n_layers, int32_t n_kv_heads, int32_t layer, const void *q, int32_t n_q_heads,
    const int32_t *q_pos, const int32_t *cache_len, float scale, float *out, int32_t *err_flag,
    hipStream_t stream) {
  prcr::DecodeParams p;
  size_t need = 0;
  prcr_status st = prcr::prepare_decode(rope, cache, dtype, batch, n_layers, n_kv_heads, layer, q,
                                        n_q_heads, q_pos, cache_len, scale, out, err_flag, &p, &need);
  if (st != PRCR_OK) return st;
  if (need > kScratchBytes) return PRCR_ERR_SCRATCH;
  // The kernels run on the stream's GPU (the current GPU for the null stream).
  int dev = -1;
  const hipError_t e = stream != nullptr ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return PRCR_ERR_HIP;
  st = scratch_for(dev, &p.ws);
  if (st != PRCR_OK) return st;
  return prcr::launch_status(prcr::launch_decode(p, dtype, rope->head_dim, cache->paged != 0, stream));
}
