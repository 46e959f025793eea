// The library's own scratch for art_decode_attention_static (include/art.h):
// a file-scope device array that stands in for the caller's workspace, so
// that the call allocates nothing.
//
// Each GPU the library runs on holds its own copy of the array from the
// module's load until the process ends.  In host code the array's name is
// not a device address: its address on the current device comes from
// hipGetSymbolAddress, taken once per device (with that device current) and
// kept; only that pointer is ever handed to a kernel.  The array is filled
// with zeros once per device at the same time, on the caller's stream.  The
// decode kernel tags everything it leaves there with the call's epoch, so
// nothing needs clearing between calls, whatever shape the previous call on
// the device had.
#include <hip/hip_runtime.h>

#include <mutex>

#include "art.h"
#include "art_internal.h"

namespace art {
namespace {

constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[ART_STATIC_SCRATCH_BYTES];

std::mutex g_mutex;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device (null until set up)

}  // namespace

int static_scratch(hipStream_t stream, void** ptr) {
  *ptr = nullptr;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    if (!p) return (int)hipErrorInvalidSymbol;
    const int z = launch_fill_zero(p, ART_STATIC_SCRATCH_BYTES, stream);
    if (z != (int)hipSuccess) return z;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return (int)hipSuccess;
}

}  // namespace art
