// tss_verify_static: the verify step with its workspace in a static device
// array that the library holds on each GPU, for callers that cannot allocate
// device memory.  The array lives in this file, and so does the lookup of its
// device address: host code never passes the array's name to a kernel or a
// copy, only the address hipGetSymbolAddress returns for the current device.
#include "../../include/tss.h"
#include "tss_internal.h"

#include <mutex>

// One copy per GPU the library runs on, held until the process ends.
static __device__ __align__(256) uint8_t scratch[TSS_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `dev`, which must be the current device;
// looked up once per device.
hipError_t scratch_on(int dev, uint8_t** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = (uint8_t*)p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" int tss_verify_static(tss_ctx* c, int32_t seq, const int32_t* draft_tokens, const int32_t* tree_parent,
                                 int32_t n_nodes, const uint8_t* skip_mask, uint32_t flags, int32_t* accept_len,
                                 int32_t* next_token) {
  if (!c) return TSS_EINVAL;
  int dev = 0;
  int r = tss::static_prepare(c, seq, &dev);
  if (r) return r;
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
  if (e != hipSuccess) return tss::static_hip_fail(c, e, "selecting the context's device");
  uint8_t* base = nullptr;
  e = scratch_on(dev, &base);
  if (e != hipSuccess) {
    if (cur != dev) (void)hipSetDevice(cur);
    return tss::static_hip_fail(c, e, "static scratch address");
  }
  r = tss::verify_in_workspace(c, base, seq, draft_tokens, tree_parent, n_nodes, skip_mask, flags, accept_len,
                               next_token);
  if (cur != dev) (void)hipSetDevice(cur);
  return r;
}
