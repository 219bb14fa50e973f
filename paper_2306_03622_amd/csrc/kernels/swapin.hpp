// Layer kernels that also move a model's weights into the arena (kept apart from the
// declarations of the plain layer kernels in kernels.hpp).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace tp {
namespace k {

// The first fp32 linear layer of a model still in pinned host memory, fused with the copy of
// the model's whole image (img_bytes, a multiple of 16) from device-visible host memory img_host
// to the device extent img_dev: y = act(x W^T + b) with W [N][K] at byte w_off and b [N] at
// b_off of the image, read from the host copy; afterwards img_dev holds every byte of the image.
// M <= 8, K % 4 == 0, K <= 1024, w_off % 16 == 0; same results as linear_f32.
hipError_t linear_f32_swap(const float* x, int M, int K, int N, int act, float* y, const void* img_host,
                           void* img_dev, uint64_t img_bytes, uint64_t w_off, uint64_t b_off, hipStream_t s);

}  // namespace k
}  // namespace tp
