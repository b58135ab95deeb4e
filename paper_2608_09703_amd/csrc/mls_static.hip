// Speculative verification with no allocation: the same launches as
// mls_spec_verify, with the per-row distribution records kept in a fixed
// device array that the library holds for the life of the process instead of
// a caller-provided workspace (for callers that cannot allocate device memory:
// code under HIP graph capture, tight serving loops).
//
// The array is a file-scope __device__ object. Host code never uses its name
// as an address (that is a host-side stand-in): its device address is looked
// up once per device with hipGetSymbolAddress, with that device current, and
// cached per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "mls.h"
#include "mls_launch.h"

namespace {

constexpr size_t kScratchBytes = (size_t)MLS_SPEC_VERIFY_STATIC_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's copy of `scratch` (looked up on the first call).
mls_status scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return mls::set_error(MLS_HIP_ERROR, "hipGetDevice failed", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return mls::set_error(MLS_UNSUPPORTED, "device index beyond the static scratch table", "");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return mls::set_error(MLS_HIP_ERROR, "hipGetSymbolAddress(scratch) failed",
                            e != hipSuccess ? hipGetErrorString(e) : "null address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MLS_OK;
}

}  // namespace

extern "C" mls_status mls_spec_verify_noalloc(const mls_sampling* s, int64_t batch, int64_t gamma,
                                              const float* draft_logits, const float* target_logits,
                                              const int32_t* draft_tokens, const float* u_accept,
                                              const float* u_sample, const void* draft_params,
                                              int32_t* n_accepted, int32_t* next_token,
                                              void* stream) {
  size_t need = 0;
  mls_status st = mls_spec_verify_workspace(batch, gamma, &need);
  if (st != MLS_OK) return st;
  if (need > kScratchBytes)
    return mls::set_error(MLS_INVALID_ARG,
                          "batch x (2 gamma + 1) distribution records exceed the static scratch "
                          "(use mls_spec_verify with a workspace)",
                          "");
  void* ws = nullptr;
  if (s && !s->greedy) {  // greedy verification reads no records
    st = scratch_on_current_device(&ws);
    if (st != MLS_OK) return st;
  }
  // The records are written by the row-parameter launch before the verify
  // launch reads them, so nothing needs clearing between calls.
  return mls_spec_verify(s, batch, gamma, draft_logits, target_logits, draft_tokens, u_accept,
                         u_sample, draft_params, n_accepted, next_token, ws, ws ? kScratchBytes : 0,
                         stream);
}
