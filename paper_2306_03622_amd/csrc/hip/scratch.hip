// The static workspace of tp_infer_noalloc: a file-scope device array that the code object
// brings with it, so requests that use it need no device allocation at all. Every device
// the library runs on holds its own copy (allocated when the code object is loaded there)
// until the process ends. Host code never names the array in a kernel argument or copy:
// its host-side symbol is only a handle. Its device address is resolved once per device,
// with that device current (scratch_init, called by tp_create), and that address is what
// the requests use.
#include <hip/hip_runtime.h>

#include <mutex>
#include <unordered_map>

#include "scratch.hpp"

static __device__ __align__(256) char scratch[tp::kNoAllocScratchBytes];

namespace {

std::mutex mu;
std::unordered_map<int, char*> resolved;   // device -> device address of `scratch`

}  // namespace

namespace tp {

hipError_t scratch_init(int device) {
  std::lock_guard<std::mutex> lk(mu);
  if (resolved.count(device)) return hipSuccess;
  int cur = -1;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  if (cur != device) return hipErrorInvalidDevice;      // the caller makes `device` current
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!ptr || reinterpret_cast<uintptr_t>(ptr) % 256) return hipErrorInvalidSymbol;
  resolved[device] = static_cast<char*>(ptr);
  return hipSuccess;
}

char* scratch_region(int device) {
  std::lock_guard<std::mutex> lk(mu);
  auto it = resolved.find(device);
  return it == resolved.end() ? nullptr : it->second;
}

}  // namespace tp
