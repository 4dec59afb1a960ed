// Device scratch of the entry point that allocates nothing.
//
// Callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops, harnesses that forbid hipMalloc) run the relational
// part of a query through aiq_run_relational_static, whose counters,
// look-back words and join hash table live in this fixed array instead of a
// caller workspace.  Each GPU the library runs on holds its own copy until
// the process ends.  In host code the array's name is only a host-side
// stand-in: its device address comes from hipGetSymbolAddress, taken once per
// device with that device current, and only that address is handed to
// kernels.  Every call on a GPU shares that GPU's array, so calls that
// overlap on one GPU race; each call clears what must start at zero.
#include <mutex>

#include "aiq_internal.h"

namespace aiq {

static __device__ __align__(256) unsigned char scratch[STATIC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
void* g_ptr[MAX_DEVICES];
std::mutex g_mu;
}  // namespace

hipError_t static_scratch(void** ptr, size_t* bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p || reinterpret_cast<uintptr_t>(p) % 256) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  *bytes = STATIC_SCRATCH_BYTES;
  return hipSuccess;
}

}  // namespace aiq
