// The layer-chain driver for callers that cannot allocate device memory:
// ifq_run_stack with its workspace (the work slots between layers) taken
// from an array of this library that every GPU it runs on holds for the
// whole process, instead of a buffer the caller allocates.
#include <hip/hip_runtime.h>

#include <mutex>

#include "ifq.h"
#include "ifq_internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;

// Device memory of the work slots. In host code this name stands for the
// array but is not its device address: only the address looked up below
// (per device) is ever passed on.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch_ptr[kMaxDevices];   // device address of scratch, per device

// The device address of scratch on the current device, looked up once per
// device with that device current.
ifq_status scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return ifq::set_error(IFQ_ERR_HIP, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return ifq::set_error(IFQ_ERR_UNSUPPORTED, "run_stack_static: device index out of range");
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return ifq::set_error(IFQ_ERR_HIP, e != hipSuccess ? hipGetErrorString(e)
                                                         : "run_stack_static: no scratch address");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return IFQ_OK;
}

}  // namespace

extern "C" {

IFQ_API size_t ifq_static_workspace_bytes(void) { return kScratchBytes; }

IFQ_API ifq_status ifq_run_stack_static(const ifq_stack* s, const void* x, void* y,
                                        hipStream_t stream) {
  if (!s) return ifq::set_error(IFQ_ERR_INVALID_ARGUMENT, "stack is NULL");
  const size_t need = ifq_stack_workspace_bytes(s);
  if (need > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof(msg),
             "run_stack_static: the stack needs %zu bytes of workspace, the static "
             "workspace holds %zu",
             need, kScratchBytes);
    return ifq::set_error(IFQ_ERR_INSUFFICIENT_BUFFER, msg);
  }
  void* ws = nullptr;
  const ifq_status st = scratch_ptr(&ws);
  if (st != IFQ_OK) return st;
  // ifq_run_stack validates the stack (again) before any launch and
  // launches nothing but the layers' kernels: no allocation, no memset
  return ifq_run_stack(s, x, y, ws, kScratchBytes, stream);
}

}  // extern "C"
