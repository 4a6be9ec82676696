// noalloc.hip -- ebd_attend_certify_noalloc: the certified decode step for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid allocation).  It runs the same kernels as ebd_attend_certify; their workspace (the
// per-(unit, head block) diagnostic counts and, for units cut into several splits, the split
// records) is a fixed array of this file instead of a caller buffer.
//
// The array is a file-scope device variable: the runtime gives every GPU that loads the library
// its own copy, zero-filled, and keeps it until the process ends.  In host code its name is only
// a host-side stand-in, never a device address: the address of the current device's copy comes
// from hipGetSymbolAddress, looked up on the first call on that device and kept per device.
// Nothing in it needs clearing between calls: the kernels zero the diagnostic counts themselves,
// and every split record the finalize reads was written earlier in the same call.  All calls on
// one GPU share its copy, so calls that overlap on one GPU (several streams, several host
// threads) race; issue them in order on one stream.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ebd.h"
#include "ebd_internal.hpp"

namespace {

constexpr size_t kScratchBytes = EBD_NOALLOC_SCRATCH_BYTES;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (looked up once per device, with that device current).
ebd_status device_scratch(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return EBD_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return EBD_ERR_HIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return EBD_OK;
}

}  // namespace

extern "C" ebd_status ebd_attend_certify_noalloc(const ebd_attend_params *p, const uint16_t *q,
                                                 const uint16_t *Kc, const uint16_t *Vc,
                                                 const float *pic, const int32_t *count, float *y,
                                                 float *vhat, float *lse, float *brange,
                                                 float *radius, uint32_t *status, void *stream) {
  size_t need = 0;
  const ebd_status cs = ebd::attend_check(p, q, Kc, Vc, pic, count, y, vhat, lse, &need);
  if (cs != EBD_OK || p->num_units == 0) return cs;
  if (need > kScratchBytes) return EBD_ERR_UNSUPPORTED;
  const ebd_status ds = ebd::device_ok();
  if (ds != EBD_OK) return ds;
  void *ws = nullptr;
  const ebd_status ss = device_scratch(&ws);
  if (ss != EBD_OK) return ss;
  return ebd::attend_launch(p, q, Kc, Vc, pic, count, y, vhat, lse, brange, radius, status, ws,
                            stream, false);
}
