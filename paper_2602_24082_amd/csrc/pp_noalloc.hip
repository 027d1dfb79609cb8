// pp_attn_fwd_noalloc: the attention forward (Sec. 3.2) for callers that cannot
// allocate device memory -- code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation.  It runs the kernels of pp_attn_fwd on the
// same plan; the plan's metadata, which pp_attn_fwd keeps in the caller's
// workspace, goes into a file-scope device array instead.
//
// Each device that runs this entry point holds its own copy of the array until
// the process ends.  Its address is looked up once per device (with that device
// current) and kept; host code passes that address to the kernels, never the
// array's name, which in host code is only a stand-in for the symbol.  Every
// call on a device reuses that device's array, so calls that overlap on one
// device (on different streams, or from several host threads without ordering)
// race on it; calls ordered on one stream do not.

#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/pp_attn.h"
#include "pp_launch.h"

namespace {

static __device__ __align__(256) uint8_t scratch[PP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of the current device's scratch, looked up on first use.
pp_status scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return pp::report_hip_error(e, "hipGetDevice (no-alloc scratch)");
  if (dev < 0 || dev >= kMaxDevices)
    return pp::report_error(PP_ERR_UNSUPPORTED, "device %d is beyond the %d devices the static scratch serves", dev,
                            kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return pp::report_hip_error(e, "hipGetSymbolAddress (no-alloc scratch)");
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return PP_OK;
}

}  // namespace

extern "C" pp_status pp_attn_fwd_noalloc(const pp_pack_desc* desc, int hq, int hkv, int head_dim, float scale,
                                         const void* q, const void* k, const void* v, void* o, float* lse,
                                         void* hip_stream) {
  return pp::attn_fwd_fixed_scratch(desc, hq, hkv, head_dim, scale, q, k, v, o, lse, PP_NOALLOC_SCRATCH_BYTES,
                                    scratch_address, (hipStream_t)hip_stream);
}
