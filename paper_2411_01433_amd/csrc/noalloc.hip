// Static device scratch of the allocation-free decode entry point.
//
// The array below is the workspace of moe_decode_step_noalloc: one copy per
// GPU, created when the library's code object is loaded on that device and
// held until the process ends.  Host code never uses the array's name as an
// address (on the host it is only a stand-in symbol): the device address is
// looked up once per device with hipGetSymbolAddress, with that device
// current, and kept here; kernels receive that address as an argument.
#include <mutex>

#include "moe_internal.h"

namespace moe {
constexpr size_t kScratchBytes = size_t(8) << 20;
}

static __device__ __align__(256) unsigned char scratch[moe::kScratchBytes];

namespace moe {

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

size_t scratch_bytes() { return kScratchBytes; }

hipError_t scratch_setup(int device, void** out) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;  // the caller makes it current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = p;
  }
  if (out) *out = g_scratch_ptr[device];
  return hipSuccess;
}

}  // namespace moe
