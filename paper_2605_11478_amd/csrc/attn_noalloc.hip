// Library-owned scratch memory for fibq_attn_decode_noalloc: the attention
// workspace (rotated-query operands, the binary16 codebook table, per-group
// tables and the split-K partial records) taken from one fixed device array
// instead of a caller allocation, for callers that cannot allocate.
//
// `scratch` is a file-scope device array.  In host code its name is only a
// stand-in for the symbol, not a device address, so the address is looked up
// once per device with hipGetSymbolAddress (with that device current) and
// kept; every later use goes through that pointer.  Each GPU that runs the
// library holds its own copy until the process ends.
#include <hip/hip_runtime.h>

#include <mutex>

#include "fibq.h"
#include "fibq_internal.h"

namespace fibq {
namespace dev {

namespace {

constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[FIBQ_ATTN_SCRATCH_BYTES];

std::mutex g_mu;
void* g_ptr[kMaxDevices];

}  // namespace

int static_attn_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDevices) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return e != hipSuccess ? (int)e : (int)hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return 0;
}

}  // namespace dev
}  // namespace fibq
