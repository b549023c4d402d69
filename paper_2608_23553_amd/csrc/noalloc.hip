// noalloc.hip - the fixed scratch of chimera_search_noalloc: a file-scope
// device array, one copy per GPU, whose device address is looked up once per
// device and kept.
//
// In host code the array's name stands for a host-side shadow, not for
// device memory: only the address returned by hipGetSymbolAddress (with the
// device current) may be handed to kernels or copies.
#include <mutex>

#include "internal.h"

namespace chimera {

static __device__ __align__(256) char scratch[kFixedScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_addr[kMaxDevices] = {};
}  // namespace

int fixed_scratch(int device, void **ptr) {
  if (device < 0 || device >= kMaxDevices) return fail(CHIMERA_E_UNSUPPORTED, "device %d: at most %d devices", device,
                                                        kMaxDevices);
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_addr[device]) {
    // the caller has made `device` current; this GPU's copy of the array
    void *p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol, "fixed scratch address");
    g_addr[device] = p;
  }
  *ptr = g_addr[device];
  return CHIMERA_OK;
}

}  // namespace chimera
