// Fixed device scratch for painn_forward_noalloc: the forward's workspace
// (features, radial basis rows, edge info, head grouping) carved from one
// file-scope device array instead of memory the library allocates, for
// callers that cannot allocate (code under graph capture, tight serving
// loops).  Each device holds its own copy of the array from the first load
// of this library's code on it until the process ends.
#include <mutex>

#include "internal.h"

static __device__ __align__(256) unsigned char scratch[NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int MAX_DEVICES = 64;
std::mutex g_mutex;
void* g_ptr[MAX_DEVICES] = {};
hipError_t g_status[MAX_DEVICES] = {};
bool g_done[MAX_DEVICES] = {};

}  // namespace

// Look up this device's address of `scratch`, once per device, with the
// device current (the caller has made it current).  In host code the
// array's name stands for a host-side shadow, not device memory: only the
// address returned here may be handed to kernels or copies.
hipError_t noalloc_scratch_init(int device) {
  if (device < 0 || device >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_done[device]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) {
      (void)hipGetLastError();
      p = nullptr;
    }
    g_ptr[device] = p;
    g_status[device] = e;
    g_done[device] = true;
  }
  return g_status[device];
}

void* noalloc_scratch(int device) {
  if (device < 0 || device >= MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lock(g_mutex);
  return g_done[device] ? g_ptr[device] : nullptr;
}
