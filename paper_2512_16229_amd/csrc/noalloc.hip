// lopa_verify_forward_noalloc: the verify forward with its working buffers in
// a file-scope device array instead of memory the library allocates, for
// callers that cannot allocate device memory where they run the step.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/lopa.h"
#include "verify.h"

namespace {

constexpr int MAX_DEVICES = 64;

// The shared working memory. Each GPU holds its own copy for the life of the
// process. In host code `scratch` names a host-side stand-in, not the device
// address: the address is taken once per device with hipGetSymbolAddress and
// only that pointer is used.
static __device__ __align__(256) unsigned char scratch[LOPA_NOALLOC_MAX_BYTES];

std::mutex g_mu;
void* g_ptr[MAX_DEVICES] = {};

int scratch_on_device(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (dev < 0 || dev >= MAX_DEVICES)
    return lopa_fail(LOPA_EHIP, "device %d outside [0, %d)", dev, MAX_DEVICES);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return lopa_fail(LOPA_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                       hipGetErrorString(e));
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return LOPA_OK;
}

}  // namespace

extern "C" int lopa_verify_forward_noalloc(const lopa_model* m, lopa_kv* kv, int32_t prefix_len,
                                           const int32_t* branch_tokens, int32_t n_branches,
                                           int32_t L, float* conf, int32_t* pred, void* stream) {
  int rc = verify_check(m, kv, prefix_len, branch_tokens, n_branches, L, conf, pred);
  if (rc) return rc;
  const size_t need = verify_ws_bytes(m, n_branches, L);
  if (need > (size_t)LOPA_NOALLOC_MAX_BYTES)
    return lopa_fail(LOPA_ESHAPE,
                     "lopa_verify_forward_noalloc: %d branches x %d rows need %zu bytes of "
                     "working memory, more than its fixed %zu",
                     n_branches, L, need, (size_t)LOPA_NOALLOC_MAX_BYTES);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return lopa_fail(LOPA_EHIP, "no current HIP device");
  if (dev != model_device(m))
    return lopa_fail(LOPA_EINVAL, "the current device %d is not the model's device %d", dev,
                     model_device(m));
  void* base = nullptr;
  if ((rc = scratch_on_device(dev, &base))) return rc;
  const VerifyWs ws = verify_ws_carve(m, n_branches, L, (char*)base);
  // the array keeps the last call's contents: the padding columns the GEMMs
  // read must be zero again (every other buffer is written before it is read)
  if ((rc = verify_ws_clear_padding(m, n_branches, L, ws, (hipStream_t)stream))) return rc;
  return verify_with_ws(m, kv, prefix_len, branch_tokens, n_branches, L, conf, pred, stream, ws);
}
