// Library-owned device scratch for caddtree_build_noalloc: the top-K table that
// caddtree_build otherwise carves out of the caller's workspace.
//
// The array lives in the code object, so each GPU the library runs on holds its
// own copy until the process ends, at its own address.  Host code never passes
// the array's name to a kernel or a copy (on the host that name is only a
// stand-in): the address is taken once per device with hipGetSymbolAddress, with
// that device current, and kept here.

#include <mutex>

#include <hip/hip_runtime.h>

#include "internal.h"

namespace caddtree {
namespace {

static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_scratch_init(int device) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[device] != nullptr) return hipSuccess;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (p == nullptr) return hipErrorInvalidSymbol;
  g_ptr[device] = p;
  return hipSuccess;
}

void* noalloc_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_mu);
  return g_ptr[device];
}

}  // namespace caddtree
