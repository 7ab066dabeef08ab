// A handle whose workspace is a file-scope device array instead of caller
// memory: for callers that cannot allocate device memory (code under HIP
// graph capture, serving loops and harnesses that forbid hipMalloc).
//
// The array is created with the code object on every device the library runs
// on and lives until the process ends.  Its device address is taken once per
// device, at the first t2i_dit_init_static on that device, with
// hipGetSymbolAddress; host code passes only that address on (the array's
// name in host code is a host-side stand-in, not a device address).  The
// workspace needs no clearing between calls: every kernel of a step writes
// each workspace element it later reads within the same call.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/t2i_dit.h"

namespace {

constexpr size_t kScratchBytes = T2I_STATIC_WORKSPACE_BYTES;
static_assert(kScratchBytes % 256 == 0, "workspace size");

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device
std::mutex g_scratch_mu;

}  // namespace

extern "C" t2i_status t2i_dit_init_static(const t2i_dit_config* cfg, const void* const* weights,
                                          void* stream, t2i_dit** out) {
  if (!out) return T2I_ERR_INVALID_ARG;
  *out = nullptr;
  const size_t need = t2i_dit_workspace_bytes(cfg);
  if (need == 0) return T2I_ERR_INVALID_ARG;             // bad config
  if (need > kScratchBytes) return T2I_ERR_WORKSPACE;    // beyond the static maximum
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return T2I_ERR_DEVICE;
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
      void* p = nullptr;
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
        (void)hipGetLastError();
        return T2I_ERR_DEVICE;
      }
      g_scratch_ptr[dev] = p;
    }
    ptr = g_scratch_ptr[dev];
  }
  return t2i_dit_init(cfg, weights, ptr, kScratchBytes, stream, out);
}
