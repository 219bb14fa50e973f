// The cache touch of warm requests (kept apart from the per-layer kernels declared in
// kernels.hpp).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace tp {
namespace k {

// Reads `bytes` (multiple of 16, 16-byte aligned) at `p` and discards them, pulling them
// into the caches; `sink` (64 words of device memory) is written only if the XOR of a
// thread's data equals a fixed constant. hipErrorInvalidValue for a null or misaligned
// argument; the launch's own error otherwise.
hipError_t touch(const void* p, uint64_t bytes, uint32_t* sink, hipStream_t s);

}  // namespace k
}  // namespace tp
