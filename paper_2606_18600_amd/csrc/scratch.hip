// The library's static device scratch array: the workspace of the decode
// entry point that allocates nothing (stage_decode_noalloc). Each GPU the
// library runs on holds its own copy of the array, at its own address, from
// the loading of the code object until the process ends.
//
// In host code the array's name is only a stand-in for the device symbol:
// its address must be looked up per device with hipGetSymbolAddress (below)
// and only that looked-up pointer is passed to kernels and copies.
#include <hip/hip_runtime.h>

#include <mutex>

#include "kernels.hpp"

static __device__ __align__(256) char scratch[stage_k::kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_addr[kMaxDevices] = {};

}  // namespace

namespace stage_k {

hipError_t static_scratch(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device) return hipErrorInvalidDevice;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_addr[device] = p;
  }
  *ptr = g_addr[device];
  return hipSuccess;
}

}  // namespace stage_k
