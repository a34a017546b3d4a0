// Allocation-free CROWN entry point: vcr_crown_bounds (without splits) run in a fixed
// device scratch array instead of the context's workspace, for callers that cannot
// allocate device memory during the call (code under HIP graph capture, serving loops).
//
// The scratch is one file-scope device array per GPU, SCRATCH_BYTES long, held by the
// process from the library's load on that device until it exits.  Its device address is
// resolved once per device (with that device current) by vcr_create and kept per device;
// host code only ever uses that address, never the array's name.  Every call on a device
// shares the device's array and finds the previous call's contents, so a call first clears
// the part its plan uses; calls that overlap on one device (two streams, two threads,
// two contexts) race on it.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ctx.h"

namespace {

constexpr size_t SCRATCH_BYTES = VCR_NOALLOC_SCRATCH_BYTES;   // 256 MiB per device
constexpr int MAX_DEVICES = 64;

static __device__ __align__(256) char scratch[SCRATCH_BYTES];

std::mutex g_mu;
char *g_addr[MAX_DEVICES] = {};   // device address of `scratch` on each device, once resolved

}  // namespace

namespace vcr {

vcr_status noalloc_setup(vcr_ctx *c) {
  if (c->device < 0 || c->device >= MAX_DEVICES) return fail(c, VCR_ERR_DEVICE, "device id out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[c->device]) {
    HIP_TRY(c, hipSetDevice(c->device));
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(c, VCR_ERR_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_addr[c->device] = static_cast<char *>(p);
  }
  c->scratch = g_addr[c->device];
  c->scratch_bytes = SCRATCH_BYTES;
  return VCR_OK;
}

}  // namespace vcr

extern "C" vcr_status vcr_crown_bounds_noalloc(vcr_ctx *c, const float *x0, int32_t B, float eps, const float *C,
                                               int32_t m, float *lb, float *ub) {
  if (!c) return VCR_ERR_ARG;
  return vcr::crown_bounds_in(c, x0, B, eps, C, m, lb, ub, c->scratch, c->scratch_bytes);
}
