// The static workspace of tp_infer_noalloc (scratch.hip).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace tp {

// Size of the static workspace: enough for BERT-base at batch 8 (48.5 MiB), the 24 x 4096
// MLP at batch 32 (32.5 MiB) or ResNet-50 at batch 2 (47.3 MiB).
constexpr uint64_t kNoAllocScratchBytes = 64ull << 20;

// Resolves the device address of the static workspace on `device`, which must be the
// current device; once per device (later calls return at once).
hipError_t scratch_init(int device);

// The address scratch_init resolved for `device`, or null if it has not succeeded there.
char* scratch_region(int device);

}  // namespace tp
