// mk_run_noalloc: mk_run with the workspace taken from a library-owned static
// device array instead of a caller buffer, for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc).
//
// `scratch` is a file-scope __device__ array: every device the library runs
// on holds its own copy, at its own address, until the process ends.  In host
// code the array's name is only a host-side stand-in, so its device address
// is looked up once per device (hipGetSymbolAddress, with that device
// current) and only that address is ever handed to kernels.  Every call on a
// device shares that device's array and it keeps the last call's contents;
// no kernel of a composition reads workspace bytes it did not write in the
// same run, so nothing needs clearing.  Calls that overlap on one device race.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "../../include/mk.h"
#include "plan.hpp"

namespace {

__device__ __align__(256) char scratch[MK_NOALLOC_WS_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];   // device address of `scratch` per device, once looked up

}  // namespace

extern "C" mk_status mk_run_noalloc(mk_module* m, const void* const* dev_inputs, void* dev_out,
                                    void* stream) {
  if (!m) return mk::fail(MK_E_INVALID_ARG, "null module");
  int64_t need = 0;
  mk_status s = mk_workspace_size(m, &need);
  if (s != MK_OK) return s;
  if (need > (int64_t)MK_NOALLOC_WS_BYTES)
    return mk::fail(MK_E_WORKSPACE, "mk_run_noalloc: the module needs " + std::to_string(need) +
                                        " workspace bytes; the static workspace holds " +
                                        std::to_string((int64_t)MK_NOALLOC_WS_BYTES));
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return mk::fail(MK_E_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return mk::fail(MK_E_UNSUPPORTED, "mk_run_noalloc: device id " + std::to_string(dev));
  void* ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
      void* p = nullptr;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return mk::fail(MK_E_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                      hipGetErrorString(e));
      g_ptr[dev] = p;
    }
    ws = g_ptr[dev];
  }
  return mk_run(m, dev_inputs, dev_out, ws, (int64_t)MK_NOALLOC_WS_BYTES, stream, nullptr);
}
