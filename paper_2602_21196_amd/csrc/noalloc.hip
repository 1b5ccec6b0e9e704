// Attention forward without any device allocation: the workspace is a
// file-scope device array instead of a caller-allocated buffer.
//
// The array is a fixed-size static, so the call needs no hipMalloc and no
// workspace argument.  Its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and kept; host code never
// passes the array's own name to a kernel, copy or memset (in host code that
// name is a host-side stand-in, not a device address).  The forward's
// workspace needs no clearing: every byte a kernel reads in it was written
// earlier in the same call (packed rows and their zero padding, the chunk
// output, the split lse rows), so what a previous call left there is never
// seen.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/upipe.h"
#include "api_internal.h"

namespace upipe {

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up on the first
// call there; UPIPE_ERR_HIP if the lookup fails, UPIPE_ERR_INVALID_ARG if
// `stream` belongs to another device (the kernels would run there with this
// device's scratch address).
int scratch_on_current_device(hipStream_t stream, char** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return UPIPE_ERR_HIP;
  hipDevice_t sdev = -1;
  if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return UPIPE_ERR_HIP;
  if (sdev != dev) return UPIPE_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return UPIPE_ERR_HIP;
    g_scratch_ptr[dev] = static_cast<char*>(p);
  }
  *out = g_scratch_ptr[dev];
  return UPIPE_OK;
}

}  // namespace

}  // namespace upipe

using namespace upipe;

extern "C" {

size_t upipe_attn_fwd_noalloc_scratch_bytes(void) { return kScratchBytes; }

int upipe_attn_fwd_noalloc(const void* q, const void* k, const void* v, void* o, float* lse,
                           int64_t S, int Hq, int Hkv, int d, int causal, int U,
                           hipStream_t stream) {
  try {
    int rc = check_attn_shape(S, Hq, Hkv, d, U);
    if (rc != UPIPE_OK) return rc;
    if (causal != 0 && causal != 1) return UPIPE_ERR_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse))
      return UPIPE_ERR_INVALID_ARG;
    if (plan_attn_fwd(S, Hq, Hkv, U).total > kScratchBytes) return UPIPE_ERR_WORKSPACE;
    char* ws = nullptr;
    rc = scratch_on_current_device(stream, &ws);
    if (rc != UPIPE_OK) return rc;
    return run_attn_fwd((const bf16*)q, (const bf16*)k, (const bf16*)v, (bf16*)o, lse, S, Hq,
                        Hkv, causal, U, ws, stream);
  } catch (...) {
    return UPIPE_ERR_HIP;
  }
}

}  // extern "C"
