// noalloc.hip - favor_attn_both_noalloc: favor_attn_both with its workspace in
// a static device array instead of caller memory, for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid hipMalloc).
//
// The array is file-scope device memory of the library's code object: every
// GPU the library runs on holds its own copy (kScratchBytes) from the moment
// the code object is loaded there until the process ends. Its device address
// is looked up once per device, with that device current, through
// hipGetSymbolAddress, and kept per device; host code passes only that address
// (never the array's own name, a host-side stand-in) to the kernels. Nothing
// here calls hipMalloc or hipFree, and favor_attn_both allocates nothing.
// The kernels need no cleared workspace, so nothing is zeroed between calls.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <mutex>

#include "../../include/favor.h"
#include "kernels.hpp"

namespace {

constexpr size_t kScratchBytes = size_t(32) << 20;   // 32 MiB per GPU
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mutex;
void *g_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array (looked up on the
// first call on that device).
favor_status scratch_ptr(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return favor::report(FAVOR_ERR_DEVICE, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return favor::report(FAVOR_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return favor::report(FAVOR_ERR_DEVICE, "hipGetSymbolAddress of the scratch array failed");
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return FAVOR_OK;
}

}  // namespace

extern "C" {

FAVOR_API size_t favor_noalloc_scratch_bytes(void) { return kScratchBytes; }

FAVOR_API favor_status favor_attn_both_noalloc(const favor_desc *g, const void *Q,
                                               const void *K, const void *V, const float *W,
                                               const float *b, void *out_bidir,
                                               void *out_causal, const float *state_in,
                                               float *state_out, float *row_scale_bidir,
                                               float *row_scale_causal, hipStream_t stream) {
  // the descriptor is validated and the size checked before any device call
  favor_status st = favor_validate_desc(g, 3);
  if (st != FAVOR_OK) return st;
  const size_t need = favor_workspace_size(g, 2);
  if (need > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof(msg),
             "the call needs %zu bytes of workspace; the static scratch holds %zu", need,
             kScratchBytes);
    return favor::report(FAVOR_ERR_WORKSPACE_TOO_SMALL, msg);
  }
  void *ws = nullptr;
  if (need > 0) {
    st = scratch_ptr(&ws);
    if (st != FAVOR_OK) return st;
  }
  return favor_attn_both(g, Q, K, V, W, b, out_bidir, out_causal, state_in, state_out,
                         row_scale_bidir, row_scale_causal, ws, need > 0 ? kScratchBytes : 0,
                         stream);
}

}  // extern "C"
