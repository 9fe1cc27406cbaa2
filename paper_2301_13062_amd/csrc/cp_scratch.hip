// cp_scratch.hip -- the library's own device scratch, for the entry point
// that allocates nothing (cp_rollout_noalloc): the temporaries of the
// unfused and concatenated levels live in one file-scope device array
// instead of a caller's workspace.  Each device the library runs on holds
// its own copy for the life of the process; its address on a device is
// looked up once, with that device current, and kept.
#include <mutex>

#include "cp_launch.h"

namespace cp {

namespace {

__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];

}  // namespace

hipError_t scratch_address(void **out) {
  *out = nullptr;
  int device = 0;
  hipError_t e = hipGetDevice(&device);
  if (e != hipSuccess) return e;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[device]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return hipSuccess;
}

}  // namespace cp
