// mt_linear_bwd_noalloc: the dense layer's backward with its workspace in a
// fixed device array of the library instead of caller memory, for callers
// that cannot allocate device memory (code under HIP graph capture, serving
// loops, harnesses that forbid hipMalloc). Same kernels and plan as
// mt_linear_bwd given a workspace of the size mt_linear_bwd_workspace reports.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>

#include "../../include/minitensor_hip.h"
#include "host.hpp"

namespace {

// One copy per GPU, alive until the process ends. Nothing in it has to start
// at zero: split-K partial tiles and db row-slice sums are written whole
// before they are read. In host code the name `scratch` stands for a
// host-side shadow, never the device memory: host code uses only the address
// hipGetSymbolAddress returns for the current device.
__device__ __attribute__((aligned(256))) char scratch[MT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` per GPU, once looked up

// The scratch array's device address on the current device (looked up on the
// first call there, with that device current).
mt_status scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return mt::host::hip_status(e);
  if (dev < 0 || dev >= kMaxDevices)
    return mt::host::fail(MT_ERR_HIP, "mt_linear_bwd_noalloc: device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return mt::host::hip_status(e);
    if (!p || ((uintptr_t)p & 255))
      return mt::host::fail(MT_ERR_HIP, "mt_linear_bwd_noalloc: unusable scratch address");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return MT_OK;
}

}  // namespace

extern "C" mt_status mt_linear_bwd_noalloc(const mt_tensor* x, const mt_tensor* w,
                                           const mt_tensor* dy, const mt_tensor* dx,
                                           const mt_tensor* dw, const mt_tensor* db,
                                           uint32_t flags, void* stream) {
  try {
    if (flags & ~MT_ACCUMULATE) return mt::host::fail(MT_ERR_INVALID, "mt_linear_bwd_noalloc: unknown flags");
    // validates every argument (host only) and sizes the plan's workspace
    size_t need = 0;
    mt_status s = mt_linear_bwd_workspace(x, w, dy, dx, dw, db, &need);
    if (s) return s;
    if (need > (size_t)MT_NOALLOC_SCRATCH_BYTES)
      return mt::host::fail(MT_ERR_WORKSPACE,
                            "mt_linear_bwd_noalloc: these sizes need " + std::to_string(need) +
                                " bytes of scratch, more than its " +
                                std::to_string((size_t)MT_NOALLOC_SCRATCH_BYTES) +
                                "-byte maximum (use mt_linear_bwd with a workspace)");
    void* ws = nullptr;
    if (need > 0) {
      const hipStream_t st = (hipStream_t)stream;
      int cur = -1;
      hipError_t e = hipGetDevice(&cur);
      if (e != hipSuccess) return mt::host::hip_status(e);
      if (st && hipGetStreamDeviceId(st) != cur)
        return mt::host::fail(MT_ERR_INVALID,
                              "mt_linear_bwd_noalloc: the stream must belong to the current device");
      if ((s = scratch_address(&ws))) return s;
    }
    return mt_linear_bwd(x, w, dy, dx, dw, db, flags, ws, need, stream);
  } catch (...) {
    return mt::host::fail(MT_ERR_INVALID, "internal error");
  }
}
