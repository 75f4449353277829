// cnn_fwd_plan_static: cnn_fwd_plan_ws with the library's own device
// scratch in place of a caller workspace, for callers that cannot allocate
// device memory (code under HIP graph capture, serving loops that forbid
// allocation).  The scratch is one file-scope device array; every GPU the
// library runs on holds its own copy until the process ends.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "internal.h"

namespace {

// Device scratch: the repacked Ker or the fp32 partial Outs of a plan
// (cnn_plan_t.ws_bytes), at most CNN_STATIC_SCRATCH_BYTES.  Its name is a
// host-side stand-in: kernels receive its device address (per device, from
// hipGetSymbolAddress), never the name.
static __device__ __align__(256) unsigned char scratch[CNN_STATIC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptr;  // device -> address of its scratch

// The scratch address on the current device, resolved once per device.
int scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return cnnlib::set_error(CNN_E_HIP, "hipGetDevice failed");
  std::lock_guard<std::mutex> g(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return CNN_OK;
  }
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !ptr)
    return cnnlib::set_error(CNN_E_HIP, "hipGetSymbolAddress of the static scratch failed");
  g_scratch_ptr[dev] = ptr;
  *out = ptr;
  return CNN_OK;
}

}  // namespace

extern "C" int cnn_fwd_plan_static(const void* In, const void* Ker, void* Out,
                                   const cnn_problem* prob, int dtype, const cnn_plan_t* plan,
                                   void* stream) {
  if (plan && plan->ws_bytes > CNN_STATIC_SCRATCH_BYTES)
    return cnnlib::set_error(CNN_E_UNSUPPORTED,
                             "plan needs more workspace than the static scratch holds "
                             "(CNN_STATIC_SCRATCH_BYTES): use cnn_fwd_plan_ws");
  // Every argument and plan check first, so an error leaves no HIP call made.
  int st = cnnlib::fwd_plan_checked(In, Ker, Out, prob, dtype, plan, nullptr,
                                    CNN_STATIC_SCRATCH_BYTES, stream, true);
  if (st != CNN_OK) return st;
  void* ws = nullptr;
  if ((st = scratch_address(&ws))) return st;
  return cnnlib::fwd_plan_checked(In, Ker, Out, prob, dtype, plan, ws, CNN_STATIC_SCRATCH_BYTES,
                                  stream, false);
}
