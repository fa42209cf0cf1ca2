// hsa_active_attention_noalloc: hsa_active_attention with its workspace taken
// from a fixed device array of this library instead of a caller buffer, for
// callers that cannot allocate device memory. See include/hsa_step.h.
//
// The array lives in the library's code object: every GPU the library is
// loaded on holds its own copy at its own address until the process ends. Its
// address on a device is looked up once (hipGetSymbolAddress, with that device
// current) and kept per device; host code uses that address, never the
// array's name. Nothing here allocates.
#include <atomic>
#include <mutex>

#include "api_util.h"

using namespace hsa_api;

namespace {

static __device__ __align__(256) unsigned char scratch[HSA_STEP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_init;

// The scratch address on the current device, or null if it cannot be found.
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_init);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (!p) {
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return nullptr;
    g_scratch[dev].store(q, std::memory_order_release);
    p = q;
  }
  return p;
}

}  // namespace

HSA_API int hsa_active_attention_noalloc(int dtype, const void* q, const void* k_cache,
                                         const void* v_cache, const int32_t* idx, int32_t n_active,
                                         int64_t n_tokens, int32_t heads, int32_t head_dim,
                                         float scale, const void* wo, void* out,
                                         hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (heads <= 0 || head_dim <= 0 || (int64_t)heads * head_dim > INT32_MAX) return HSA_STEP_ERR_SHAPE;
  if (n_active < 0 || n_tokens < 0 || n_active > n_tokens) return HSA_STEP_ERR_SHAPE;
  if (n_active == 0) return HSA_STEP_OK;
  // the compact attention output must fit; the rest of the array may hold key parts
  if (hsa_attention_workspace_bytes(dtype, n_active, heads * head_dim) >
      (size_t)HSA_STEP_NOALLOC_SCRATCH_BYTES)
    return HSA_STEP_ERR_WORKSPACE;
  void* ws = device_scratch();
  if (!ws) return HSA_STEP_ERR_LAUNCH;
  return hsa_active_attention(dtype, q, k_cache, v_cache, idx, n_active, n_tokens, heads, head_dim,
                              scale, wo, out, ws, (size_t)HSA_STEP_NOALLOC_SCRATCH_BYTES, stream);
}
